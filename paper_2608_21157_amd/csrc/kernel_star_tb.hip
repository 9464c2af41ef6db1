// kernel_star_tb.hip -- two star-stencil steps fused in one pass (temporal blocking),
// 3D, radius R <= 4, gfx950.
//
// Computes u2 = S(S(u0)) for the star operator S (centre plus -R..-1, +1..+R along z, y
// and x; cross-correlation as in the HIERA "Case-study protocol", generalised to stars,
// periodic wrap and batched volumes), reading u0 and writing u2 once, so a step costs
// half the HBM traffic of a one-step sweep.  Under the zero boundary the intermediate
// u1 is zero outside the grid, exactly as if it had been written and re-read.
//
// A workgroup owns a TXV-vector x TYW-row tile of the x-y plane and streams a chunk of
// z planes.  Two stages run in the same loop:
//   stage 1 computes u1 on the tile plus its R-row bands above and below and its
//           whole-vector bands left and right (the points stage 2 reads; the corner
//           blocks, which a star never reads, are skipped);
//   stage 2 computes u2 on the tile, R planes behind stage 1.
// One thread owns one column of the stage-1 region (a 16-byte vector along x): its u0
// z-queue (2R + 1 planes plus PF prefetched) and its u1 z-queue (2R + 1 planes) live in
// registers.  Both queues rotate through the same 2R + 1 + PF slots, so the loop is
// unrolled that many times and every register index is static.  The current u0 plane
// (stage 1's in-plane neighbours, over the stage-1 region and one more band) and the
// current u1 plane (stage 2's in-plane neighbours) are staged in LDS: double-buffered
// with one barrier per plane at radius 1 and 2, and two planes per barrier (four
// buffers) at radius 3 and 4.  Band threads use their u1 queue as the R-plane delay line
// that feeds the u1 plane stage 2 reads.
#include "common.hpp"
#include "plan.hpp"


namespace stencil {
namespace {

struct Tb2Params {
    int nz, ny, nx;
    long long vol;
    int ntx, nty;
    int zc, nzc;
    int nblocks;
    int channels;
};

template <typename T, int R, int PF>
struct Tb2Shape {
    static constexpr int VEC = Vec16<T>::N;
    static constexpr int TXV = 16;                       // tile width in vectors
    static constexpr int TYW = 32;                       // tile height in rows
    static constexpr int HXV = (R + VEC - 1) / VEC;      // x reach in vectors
    static constexpr int NTILE = TXV * TYW;
    // stage-1 bands around the tile: R rows above and below, HXV vectors left and right
    static constexpr int NBAND_TB = 2 * R * TXV;
    static constexpr int NBAND_LR = 2 * TYW * HXV;
    static constexpr int NS1 = NTILE + NBAND_TB + NBAND_LR;       // stage-1 columns
    static constexpr int THREADS = ((NS1 + 63) / 64) * 64;
    // u0 cells stage 1 reads beyond its own columns
    static constexpr int NX_TB = 2 * R * TXV;            // rows -2R..-R-1, TYW+R..TYW+2R-1
    static constexpr int NX_CORNER = 2 * R * 2 * HXV;    // x reach of the top/bottom bands
    static constexpr int NX_LR = 2 * TYW * HXV;          // x reach of the left/right bands
    static constexpr int NEXTRA = NX_TB + NX_CORNER + NX_LR;
    static constexpr int NEX = (NEXTRA + THREADS - 1) / THREADS;
    // LDS rectangles: u0 over rows -2R..TYW+2R-1, vectors -2HXV..TXV+2HXV-1;
    // u1 over rows -R..TYW+R-1, vectors -HXV..TXV+HXV-1
    static constexpr int W0 = TXV + 4 * HXV, H0 = TYW + 4 * R;
    static constexpr int W1 = TXV + 2 * HXV, H1 = TYW + 2 * R;
    // queue slots (both queues): the 2R + 1 planes of the window plus PF prefetched u0
    // planes (PF odd, so that the slot count is even)
    static constexpr int NQ = 2 * R + 1 + PF;
    // planes per barrier: two at radius 3 and 4 (one workgroup per CU in any case, so the
    // four LDS buffers cost no occupancy), one below (where the two-buffer footprint keeps
    // a second workgroup per CU)
    static constexpr bool PAIR = R >= 3;
    static constexpr int NBUF = PAIR ? 4 : 2;
    // in a pair, the second plane stages u1 of plane z1 + 1 - R before the first plane's
    // stage 1 has run: that plane must come from an earlier pair
    static_assert(!PAIR || R >= 2, "pairs need the staged u1 plane to be at least 2 behind");
    static_assert(NTILE % 64 == 0, "stage 2 must cover whole waves");
    static_assert(NQ % 2 == 0, "the extra-cell registers alternate by iteration parity");
};

// LDS vector index of tile-relative (row r, vector v) in a rectangle whose origin is
// (-oy, -ov) and pitch is w.
__device__ __forceinline__ int rect_index(int r, int v, int oy, int ov, int w)
{
    return (r + oy) * w + (v + ov);
}

template <typename T, int R, int PF, bool PERIODIC, int STORE_CP>
__global__ __launch_bounds__((Tb2Shape<T, R, PF>::THREADS)) void stencil_star_tb2_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ w, Tb2Params p)
{
    using S = Tb2Shape<T, R, PF>;
    constexpr int VEC = S::VEC, TXV = S::TXV, TYW = S::TYW, HXV = S::HXV, NQ = S::NQ;
    constexpr int E = sizeof(T);
    // Each LDS plane ends with 64 spare cells: lanes that own no cell of a plane write
    // their lane's spare cell instead, so every write is unconditional.  The loop body
    // has no branch around a global load, store or LDS write; that keeps the compiler's
    // wait counts exact, so a plane waits only for the loads it consumes and never for
    // the store and prefetches just issued.
    constexpr int SPARE0 = S::H0 * S::W0, SPARE1 = S::H1 * S::W1;
    __shared__ Vec16<T> lds0[S::NBUF][SPARE0 + 64];
    __shared__ Vec16<T> lds1[S::NBUF][SPARE1 + 64];

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

    // ---- this thread's stage-1 column (tile-relative row r, vector v) ------------------
    // Lanes past the stage-1 columns (present when the column count is not a multiple of
    // 64) compute on cell (0, 0), load nothing, store nothing and write spare cells.
    const bool col = tid < S::NS1, tile = tid < S::NTILE;
    int r = 0, v = 0;
    if (tile) {
        r = tid / TXV;
        v = tid % TXV;
    } else if (col) {
        int j = tid - S::NTILE;
        if (j < S::NBAND_TB) {
            const int k = j / TXV;
            r = k < R ? k - R : TYW + k - R;
            v = j % TXV;
        } else {
            j -= S::NBAND_TB;
            const int k = j % (2 * HXV);
            r = j / (2 * HXV);
            v = k < HXV ? k - HXV : TXV + k - HXV;
        }
    }
    const int gy = y0 + r, gx = x0 + v * VEC;
    const bool inside = col && gy >= 0 && gy < p.ny && gx >= 0 && gx < p.nx;
    const bool wave_inside = __all(inside);   // every lane of this wave
    auto goff = [&](int yy, int xx) {
        if (PERIODIC)
            return (wrap_index(yy, p.ny) * p.nx + wrap_index(xx, p.nx)) * E;
        return (yy >= 0 && yy < p.ny && xx >= 0 && xx < p.nx) ? (yy * p.nx + xx) * E
                                                               : kOutOfRange;
    };
    const int qoff = col ? goff(gy, gx) : kOutOfRange;
    const int soff = (tile && inside) ? (gy * p.nx + gx) * E : kOutOfRange;
    const int i0 = rect_index(r, v, 2 * R, 2 * HXV, S::W0);   // own cell in the u0 plane
    const int i1 = rect_index(r, v, R, HXV, S::W1);           // own cell in the u1 plane
    const int w0 = col ? i0 : SPARE0 + lane;                  // where this lane writes
    const int w1 = col ? i1 : SPARE1 + lane;

    // ---- u0 cells beyond the stage-1 columns that this thread stages ------------------
    int xoff[S::NEX], xidx[S::NEX];
#pragma unroll
    for (int h = 0; h < S::NEX; ++h) {
        int j = tid + h * S::THREADS;
        int rr = 0, vv = 0;
        bool any = true;
        if (j < S::NX_TB) {
            const int k = j / TXV;
            rr = k < R ? k - 2 * R : TYW + R + k - R;
            vv = j % TXV;
        } else if ((j -= S::NX_TB) < S::NX_CORNER) {
            const int k = j % (2 * HXV);
            const int q = j / (2 * HXV);
            rr = q < R ? q - R : TYW + q - R;
            vv = k < HXV ? k - HXV : TXV + k - HXV;
        } else if ((j -= S::NX_CORNER) < S::NX_LR) {
            const int k = j % (2 * HXV);
            rr = j / (2 * HXV);
            vv = k < HXV ? k - 2 * HXV : TXV + HXV + k - HXV;
        } else {
            any = false;
        }
        xidx[h] = any ? rect_index(rr, vv, 2 * R, 2 * HXV, S::W0) : SPARE0 + lane;
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

    // ---- z range: stage 2 writes [z0, z0 + n); stage 1 runs R planes ahead -----------
    const int z0 = zi * p.zc;
    const int n = min(p.zc, p.nz - z0);
    const int zs1 = dir > 0 ? z0 - R : z0 + n - 1 + R;  // stage-1 plane of iteration 0
    const int iters = n + 2 * R;

    // A plane outside the grid gets a zero-length resource under the zero boundary (its
    // loads return 0); periodic planes wrap.  Planes past the chunk's end are loaded
    // harmlessly by the last iterations' prefetches.
    auto plane_rsrc = [&](int z) {
        if (PERIODIC)
            return make_rsrc(src + wrap_index(z, p.nz) * plane, plane_bytes);
        // a plane outside the grid keeps its address (never dereferenced: zero records),
        // which leaves the address affine in the iteration, without a select
        const bool ok = unsigned(z) < unsigned(p.nz);  // 0 <= z < nz
        return make_rsrc(src + (long long)z * plane, ok ? plane_bytes : 0u);
    };
    auto z_inside = [&](int z) { return PERIODIC || unsigned(z) < unsigned(p.nz); };

    // ---- queues: position i of iteration m (phase m mod NQ) is slot (phase + i) mod NQ
    // q0 position i holds u0 at plane z1 + dir * (i - R), i = 0 .. 2R + PF (the last PF
    // prefetched)
    // q1 position i holds u1 at plane z2 + dir * (i - R), i = 0 .. 2R, z2 = z1 - dir * R
    // xr[k] holds the extra cells of the plane of the next iteration with parity k (NQ is
    // even, so the parity of the phase is the parity of the iteration)
    // The extra cells are loaded before the queue so that, at the loop head, as many loads
    // follow them on the entry path as in the steady state (the waits stay partial).
    Vec16<T> q0[NQ], q1[NQ], xr[2][S::NEX];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const auto rx = plane_rsrc(zs1 + dir * k);
#pragma unroll
        for (int h = 0; h < S::NEX; ++h)
            xr[k][h] = bload16<T>(rx, xoff[h]);
    }
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
        q0[i] = bload16<T>(plane_rsrc(zs1 + dir * (i - R)), qoff);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            q1[i].e[e] = T(0);
    }

    // One stencil evaluation of a column: z from its queue, y and x from the LDS plane
    // `buf`.  The in-plane operands are read in two batches, the R rows above first, then
    // the R rows below and the x neighbours; each batch is issued together before its
    // arithmetic, so its reads are in flight at the same time, and at most about half the
    // operands occupy registers at once (146 -> 131 VGPRs at radius 4, 3% faster).
    auto stencil_at = [&](const Vec16<T> *buf, int idx, int pitch, const Vec16<T> (&q)[NQ],
                          int phase) {
        Vec16<T> ga[R];
#pragma unroll
        for (int i = 0; i < R; ++i)
            ga[i] = buf[idx + (i - R) * pitch];
        T acc[VEC];
        const Vec16<T> c = q[(phase + R) % NQ];
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[e] = wz[R] * c.e[e];
#pragma unroll
        for (int i = 0; i < 2 * R + 1; ++i) {
            if (i == R)
                continue;
            const Vec16<T> u = q[(phase + i) % NQ];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wz[i], u.e[e], acc[e]);
        }
#pragma unroll
        for (int i = 0; i < R; ++i)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wy[i], ga[i].e[e], acc[e]);
        Vec16<T> gb[R + 2 * HXV];
#pragma unroll
        for (int i = 0; i < R; ++i)
            gb[i] = buf[idx + (i + 1) * pitch];
        // x: the row of scalars from HXV vectors left to HXV vectors right.  Where the
        // reach is shorter than a vector only the R elements next to the centre vector are
        // read on each side (one ds_read2 of 4 or 8 bytes per side pair instead of two
        // 16-byte reads)
        constexpr bool NARROW = HXV == 1 && R < VEC;
        T xs[(2 * HXV + 1) * VEC];
        if constexpr (NARROW) {
            const T *fb = reinterpret_cast<const T *>(buf);
#pragma unroll
            for (int e = VEC - R; e < VEC; ++e)
                xs[e] = fb[(idx - 1) * VEC + e];
#pragma unroll
            for (int e = 0; e < R; ++e)
                xs[2 * VEC + e] = fb[(idx + 1) * VEC + e];
        } else {
#pragma unroll
            for (int k = 0; k < HXV; ++k) {
                gb[R + k] = buf[idx - HXV + k];
                gb[R + HXV + k] = buf[idx + 1 + k];
            }
        }
#pragma unroll
        for (int i = 0; i < R; ++i)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wy[R + i], gb[i].e[e], acc[e]);
        if constexpr (!NARROW) {
#pragma unroll
            for (int k = 0; k < HXV; ++k) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    xs[k * VEC + e] = gb[R + k].e[e];
                    xs[(HXV + 1 + k) * VEC + e] = gb[R + HXV + k].e[e];
                }
            }
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            xs[HXV * VEC + e] = c.e[e];
#pragma unroll
        for (int i = 0; i < 2 * R; ++i) {
            const int ox = i < R ? i - R : i - R + 1;
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[e] = fma(wx[i], xs[HXV * VEC + e + ox], acc[e]);
        }
        Vec16<T> res;
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            res.e[e] = acc[e];
        return res;
    };

    // (Every lambda of the loop is forced inline: a call that stays out of line makes the
    // register queues it captures live in scratch memory, 20x slower.)
    // One iteration is split in two: `stage` writes the LDS planes of iteration m (u0 at
    // z1 with its extra cells, u1 at z2) into buffer `buf` and refills the extra-cell
    // registers; after a barrier, `compute` runs stage 1 and stage 2 of iteration m from
    // that buffer, stores u2 and prefetches the next u0 plane.
    auto stage = [&](int m, int phase, int buf) __attribute__((always_inline)) {
        const int z1 = zs1 + dir * m;
        const int par = phase & 1;
        Vec16<T> *b0 = lds0[buf];
        Vec16<T> *b1 = lds1[buf];
        // stage the u0 plane z1 (own columns and the extra cells) and the u1 plane z2,
        // then refill the extra-cell registers with plane z1 + 2 dir
        b0[w0] = q0[(phase + R) % NQ];
        b1[w1] = q1[(phase + R) % NQ];
#pragma unroll
        for (int h = 0; h < S::NEX; ++h)
            b0[xidx[h]] = xr[par][h];
        const auto rx = plane_rsrc(z1 + 2 * dir);
#pragma unroll
        for (int h = 0; h < S::NEX; ++h)
            xr[par][h] = bload16<T>(rx, xoff[h]);
    };
    auto compute = [&](int m, int phase, int buf) __attribute__((always_inline)) {
        const int z1 = zs1 + dir * m;
        const int z2 = z1 - dir * R;
        const Vec16<T> *b0 = lds0[buf];
        const Vec16<T> *b1 = lds1[buf];
        // stage 1: u1 at plane z1; zero outside the grid under the zero boundary
        Vec16<T> u1 = stencil_at(b0, i0, S::W0, q0, phase);
        // At radius 3 and 4 a wave whose columns all lie inside the grid skips the selects
        // on planes inside it (a wave-uniform branch; the common case): 0.6526 -> 0.6441
        // and 0.6548 -> 0.6492 ms per 512^3 radius-4 call, same-box A/B.  At radius 1 the
        // branch made the 256^3 ten-step call 15% slower, so there the selects stay.
        if (!PERIODIC && !(S::PAIR && wave_inside && z_inside(z1))) {
            const bool keep = inside && z_inside(z1);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                u1.e[e] = keep ? u1.e[e] : T(0);
        }
        q1[(phase + 2 * R) % NQ] = u1;
        // stage 2: u2 at plane z2 on the tile columns once the u1 queue is full (a
        // wave-uniform condition: the tile is a whole number of waves).  Reading both
        // stages' operands up front was measured slower (register pressure).
        const bool st2 = tile && m >= 2 * R;
        Vec16<T> u2;
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            u2.e[e] = T(0);
        if (st2) {
            u2 = stencil_at(b1, i1, S::W1, q1, phase);
        }
        // the resource depends on the uniform iteration only (a per-lane base would make
        // the compiler serialise the store over lanes); the offset masks the lanes
        // before stage 2 has a full queue every lane's offset is out of range, so the
        // address of plane z2 (then possibly outside the grid) is never dereferenced
        bstore16<T, STORE_CP>(make_rsrc(dst + (long long)z2 * plane, plane_bytes),
                              st2 ? soff : kOutOfRange, u2);
        // queue position 0 is free: prefetch u0 at plane z1 + dir * (R + PF + 1), first
        // used PF + 1 iterations from now
        q0[phase] = bload16<T>(plane_rsrc(z1 + dir * (R + PF + 1)), qoff);
    };

    // whole groups of NQ iterations in the loop, the remainder after it: an early exit
    // inside the loop body would merge into the loop head and make its waits conservative
    int m0 = 0;
    if constexpr (S::PAIR) {
        // two planes per barrier: both are staged first (the second plane's u0 is queued
        // and its u1 plane was computed in an earlier pair), then both are computed; the
        // pairs alternate between buffers 0-1 and 2-3.  Halving the barriers gave 797 ->
        // 818 Gpoints/s at radius 4 (same-box A/B).
        auto pair = [&](int m, int phase, bool second) __attribute__((always_inline)) {
            const int set = 2 * ((m >> 1) & 1);
            stage(m, phase, set);
            stage(m + 1, phase + 1, set + 1);
            __syncthreads();
            compute(m, phase, set);
            if (second)
                compute(m + 1, phase + 1, set + 1);
        };
        for (; m0 + NQ <= iters; m0 += NQ) {
#pragma unroll
            for (int ph = 0; ph < NQ; ph += 2)
                pair(m0 + ph, ph, true);
        }
#pragma unroll
        for (int ph = 0; ph < NQ - 1; ph += 2)
            if (m0 + ph < iters)
                pair(m0 + ph, ph, m0 + ph + 1 < iters);
    } else {
        auto step = [&](int m, int phase) __attribute__((always_inline)) {
            stage(m, phase, phase & 1);
            __syncthreads();
            compute(m, phase, phase & 1);
        };
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
}

// prefetched u0 planes per column
constexpr int kPrefetch = 1;

// Workgroups of `kernel` one CU holds at once (1 if the query fails).
template <typename K>
int blocks_per_cu(K kernel, int threads)
{
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) !=
            hipSuccess ||
        per_cu < 1)
        return 1;
    return per_cu;
}

template <typename T, int R>
Tb2Params make_params(const Geometry &g, int resident, int per_cu)
{
    using S = Tb2Shape<T, R, kPrefetch>;
    Tb2Params p{};
    p.nz = int(g.nz);
    p.ny = int(g.ny);
    p.nx = int(g.nx);
    p.vol = g.vol;
    p.ntx = int((g.nx + S::TXV * S::VEC - 1) / (S::TXV * S::VEC));
    p.nty = int((g.ny + S::TYW - 1) / S::TYW);
    p.channels = g.channels;
    const long long base = g.batch * p.ntx * p.nty;
    // one round of workgroups: as many as the GPU holds at once (measured best against
    // 1.5x, 2x and 4x that: a second round runs with a ragged tail and more chunk starts);
    // chunks of at least 8 radii so the 2R-plane start-up of stage 2 stays small
    const long long min_len = 8 * R;
    const long long max_chunks = (p.nz + min_len - 1) / min_len;
    // Where that round holds several workgroups per CU in chunks shorter than 32 planes,
    // the round is one workgroup per CU instead, in chunks twice as long or more: the
    // 2R-plane start-up is then a smaller share of each chunk (256^3, radius 1: 0.1254 ->
    // 0.1201 ms per 10-step call, 0.0250 -> 0.0240 per 2-step call; 128^3 and the 512^3
    // radius-4 grid are unaffected).  grid_scale still scales from this default.
    long long round = resident;
    if (per_cu > 1) {
        const long long n0 = std::min((resident + base - 1) / base, max_chunks);
        if (p.nz < 32 * n0)
            round = resident / per_cu;
    }
    const long long target = scaled_target(round, g.grid_scale);
    long long nzc = (target + base - 1) / base;
    if (nzc > max_chunks)
        nzc = max_chunks;
    if (nzc < 1)
        nzc = 1;
    p.zc = int((p.nz + nzc - 1) / nzc);
    p.nzc = (p.nz + p.zc - 1) / p.zc;
    p.nblocks = int(base * p.nzc);
    return p;
}

template <typename T, int R, bool PERIODIC, int CP>
hipError_t launch_bc(const Geometry &g, const void *src, void *dst, const void *w,
                     hipStream_t stream)
{
    using S = Tb2Shape<T, R, kPrefetch>;
    const auto kernel = stencil_star_tb2_kernel<T, R, kPrefetch, PERIODIC, CP>;
    static const int resident = resident_blocks(kernel, S::THREADS);
    static const int per_cu = blocks_per_cu(kernel, S::THREADS);
    const Tb2Params p = make_params<T, R>(g, resident, per_cu);
    kernel<<<dim3(p.nblocks), dim3(S::THREADS), 0, stream>>>(
        static_cast<const T *>(src), static_cast<T *>(dst), static_cast<const T *>(w), p);
    return hipGetLastError();
}

template <typename T, int R, int CP>
hipError_t launch_cp(const Geometry &g, const void *src, void *dst, const void *w,
                     hipStream_t stream)
{
    if (g.boundary == STENCIL_PERIODIC)
        return launch_bc<T, R, true, CP>(g, src, dst, w, stream);
    return launch_bc<T, R, false, CP>(g, src, dst, w, stream);
}

template <typename T, int R>
hipError_t launch_r(const Geometry &g, const void *src, void *dst, const void *w,
                    hipStream_t stream)
{
    if (streaming_stores(g))
        return launch_cp<T, R, kNonTemporal>(g, src, dst, w, stream);
    return launch_cp<T, R, 0>(g, src, dst, w, stream);
}

template <typename T>
hipError_t launch_t(const Geometry &g, const void *src, void *dst, const void *w,
                    hipStream_t stream)
{
    switch (g.radius) {
    case 1: return launch_r<T, 1>(g, src, dst, w, stream);
    case 2: return launch_r<T, 2>(g, src, dst, w, stream);
    case 3: return launch_r<T, 3>(g, src, dst, w, stream);
    case 4: return launch_r<T, 4>(g, src, dst, w, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool star_tb2_supported(const Geometry &g)
{
    return g.ndim == 3 && star_stream_supported(g);
}

hipError_t launch_star_tb2(const Geometry &g, const void *src, void *dst, const void *w,
                           hipStream_t stream)
{
    if (g.dtype == STENCIL_F32)
        return launch_t<float>(g, src, dst, w, stream);
    return launch_t<double>(g, src, dst, w, stream);
}

}  // namespace stencil
