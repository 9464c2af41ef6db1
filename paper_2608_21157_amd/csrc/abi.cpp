// abi.cpp -- the C ABI of the stencil library: argument validation, plan lifetime,
// coefficient upload and the step loop (ping-pong between `out` and the plan's grid).
//
// The operator is the iterated zero-padded cross-correlation of the HIERA case study
// (experimental setup, "Case-study protocol"), generalised as documented in stencil.h.
// Every check below runs on the host before the first HIP call of an entry point.
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include "entry.hpp"
#include "plan.hpp"

using stencil::Geometry;
using stencil::Plan;

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace stencil {

stencil_status fail(stencil_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = std::string(stencil_status_str(st)) + ": " + buf;
    return st;
}

stencil_status hip_fail(hipError_t e, const char *what)
{
    return fail(STENCIL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

void clear_error()
{
    g_last_error.clear();
}

}  // namespace stencil

using stencil::fail;
using stencil::hip_fail;

namespace {

int32_t points(int32_t shape, int32_t ndim, int32_t radius)
{
    if ((ndim != 2 && ndim != 3) || radius < 0)
        return -1;
    if (shape == STENCIL_STAR)
        return 1 + 2 * ndim * radius;
    if (shape == STENCIL_BOX) {
        int32_t side = 2 * radius + 1;
        return ndim == 2 ? side * side : side * side * side;
    }
    return -1;
}

// Largest grid handled: element offsets are 64-bit, but each volume must stay below 2^31
// elements so that in-volume indices fit the kernels' 32-bit arithmetic.
constexpr int64_t kMaxVolume = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxElements = int64_t(1) << 40;

stencil_status validate_desc(const stencil_desc *d, Geometry *g)
{
    if (d == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "desc is NULL");
    if (d->ndim != 2 && d->ndim != 3)
        return fail(STENCIL_ERR_INVALID_ARG, "ndim must be 2 or 3 (got %d)", d->ndim);
    for (int a = 0; a < d->ndim; ++a)
        if (d->dims[a] < 1)
            return fail(STENCIL_ERR_INVALID_ARG, "dims[%d] must be >= 1 (got %lld)", a,
                        (long long)d->dims[a]);
    if (d->batch < 1)
        return fail(STENCIL_ERR_INVALID_ARG, "batch must be >= 1");
    if (d->channels < 1)
        return fail(STENCIL_ERR_INVALID_ARG, "channels must be >= 1");
    if (d->dtype != STENCIL_F32 && d->dtype != STENCIL_F64)
        return fail(STENCIL_ERR_INVALID_ARG, "unknown dtype %d", d->dtype);
    if (d->shape != STENCIL_STAR && d->shape != STENCIL_BOX)
        return fail(STENCIL_ERR_INVALID_ARG, "unknown shape %d", d->shape);
    if (d->boundary != STENCIL_ZERO && d->boundary != STENCIL_PERIODIC)
        return fail(STENCIL_ERR_INVALID_ARG, "unknown boundary %d", d->boundary);
    if (d->has_coeff_field != 0 && d->has_coeff_field != 1)
        return fail(STENCIL_ERR_INVALID_ARG, "has_coeff_field must be 0 or 1");
    if (d->radius < 0)
        return fail(STENCIL_ERR_INVALID_ARG, "radius must be >= 0");
    if (d->temporal_depth < 0)
        return fail(STENCIL_ERR_INVALID_ARG, "temporal_depth must be >= 0");
    if (d->variant < STENCIL_VARIANT_AUTO || d->variant > STENCIL_VARIANT_STREAM)
        return fail(STENCIL_ERR_INVALID_ARG, "unknown variant %d", d->variant);
    if (d->tile < 0 || d->tile > 2)
        return fail(STENCIL_ERR_INVALID_ARG, "tile must be 0, 1 or 2 (got %d)", d->tile);
    if (d->grid_scale < -2 || d->grid_scale > 2)
        return fail(STENCIL_ERR_INVALID_ARG, "grid_scale must be in -2..2 (got %d)",
                    d->grid_scale);
    const int rmax = (d->shape == STENCIL_STAR) ? 4 : (d->ndim == 2 ? 4 : 3);
    if (d->radius > rmax)
        return fail(STENCIL_ERR_UNSUPPORTED, "radius %d exceeds %d for this shape", d->radius,
                    rmax);

    g->ndim = d->ndim;
    g->nz = (d->ndim == 3) ? d->dims[0] : 1;
    g->ny = (d->ndim == 3) ? d->dims[1] : d->dims[0];
    g->nx = (d->ndim == 3) ? d->dims[2] : d->dims[1];
    if (g->nz > kMaxVolume || g->ny > kMaxVolume || g->nx > kMaxVolume)
        return fail(STENCIL_ERR_UNSUPPORTED, "extent too large");
    g->vol = g->nz * g->ny * g->nx;
    if (g->vol / g->nx / g->ny != g->nz || g->vol > kMaxVolume)
        return fail(STENCIL_ERR_UNSUPPORTED, "volume exceeds 2^31-1 elements");
    if (d->batch > kMaxElements / g->vol)
        return fail(STENCIL_ERR_UNSUPPORTED, "batch * volume exceeds 2^40 elements");
    g->batch = d->batch;
    g->channels = d->channels;
    g->npts = points(d->shape, d->ndim, d->radius);
    g->shape = d->shape;
    g->radius = d->radius;
    g->boundary = d->boundary;
    g->field = d->has_coeff_field != 0;
    g->dtype = d->dtype;
    g->elt = (d->dtype == STENCIL_F32) ? 4 : 8;
    g->tile = d->tile;
    g->grid_scale = d->grid_scale;
    return STENCIL_OK;
}

bool overlaps(const void *a, const void *b, size_t bytes)
{
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + bytes && pb < pa + bytes;
}

bool aligned16(const void *p)
{
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

}  // namespace

namespace stencil {

// Host-side checks shared by the apply entry points and stencil_tune.
stencil_status check_call(const Plan *p, const void *in, const void *out, const int64_t dims[3],
                          const void *coeffs, const void *coeff_field, int32_t radius,
                          int32_t boundary, int32_t steps)
{
    const Geometry &g = p->geo;
    if (in == nullptr || out == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "in and out must be non-NULL device pointers");
    if (coeffs == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "coeffs must be a host pointer");
    if (dims == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "dims is NULL");
    if (steps < 0)
        return fail(STENCIL_ERR_INVALID_ARG, "steps must be >= 0 (got %d)", steps);
    for (int a = 0; a < g.ndim; ++a)
        if (dims[a] != p->desc.dims[a])
            return fail(STENCIL_ERR_MISMATCH, "dims[%d] = %lld, plan has %lld", a,
                        (long long)dims[a], (long long)p->desc.dims[a]);
    if (radius != g.radius)
        return fail(STENCIL_ERR_MISMATCH, "radius %d, plan has %d", radius, g.radius);
    if (boundary != g.boundary)
        return fail(STENCIL_ERR_MISMATCH, "boundary %d, plan has %d", boundary, g.boundary);
    if ((coeff_field != nullptr) != g.field)
        return fail(STENCIL_ERR_MISMATCH, g.field ? "the plan needs a coefficient field"
                                                  : "the plan has no coefficient field");
    const size_t bytes = size_t(g.batch) * size_t(g.vol) * g.elt;
    if (overlaps(in, out, bytes))
        return fail(STENCIL_ERR_ALIAS, "out overlaps in");
    if (coeff_field != nullptr && overlaps(coeff_field, out, bytes))
        return fail(STENCIL_ERR_ALIAS, "out overlaps the coefficient field");
    return STENCIL_OK;
}

bool runs_fast(const Plan *p, const void *in, const void *out, const void *coeff_field)
{
    // fast kernels use 16-byte vector accesses; misaligned pointers run the generic kernel
    return p->variant == STENCIL_VARIANT_STREAM && aligned16(in) && aligned16(out) &&
           (coeff_field == nullptr || aligned16(coeff_field));
}

int launch_count(const Plan *p, bool fast, int steps)
{
    const int depth = fast ? p->depth : 1;
    return (steps + depth - 1) / depth;
}

stencil_status enqueue_steps(const Plan *p, bool fast, const void *in, void *out,
                             const void *coeff_field, const void *w, void *grid, int steps,
                             hipStream_t stream)
{
    const Geometry &g = p->geo;
    hipError_t e;
    if (steps == 0) {
        const size_t bytes = size_t(g.batch) * size_t(g.vol) * g.elt;
        if ((e = hipMemcpyAsync(out, in, bytes, hipMemcpyDeviceToDevice, stream)) != hipSuccess)
            return hip_fail(e, "hipMemcpyAsync(copy for steps = 0)");
        return STENCIL_OK;
    }
    const int depth = fast ? p->depth : 1;
    const int launches = launch_count(p, fast, steps);
    // launch i writes `out` when an even number of launches follows it, so the last one
    // always lands in `out`; launch i > 0 reads what launch i - 1 wrote
    const void *src = in;
    int left = steps;
    for (int i = 0; i < launches; ++i) {
        const int d = left < depth ? left : depth;
        void *dst = ((launches - 1 - i) % 2 == 0) ? out : grid;
        if (fast)
            e = launch_stream(g, src, dst, coeff_field, w, d, stream);
        else
            e = launch_generic(g, src, dst, coeff_field, w, stream);
        if (e != hipSuccess)
            return hip_fail(e, "kernel launch");
        src = dst;
        left -= d;
    }
    return STENCIL_OK;
}

}  // namespace stencil

using stencil::check_call;

namespace {

// A launch configuration: what stencil_tune varies and fixes in the plan.
struct Config {
    int variant, depth, tile, grid_scale;
};

Config config_of(const Plan *p)
{
    return {p->variant, p->depth, p->geo.tile, p->geo.grid_scale};
}

void set_config(Plan *p, const Config &c)
{
    p->variant = c.variant;
    p->depth = c.depth;
    p->geo.tile = c.tile;
    p->geo.grid_scale = c.grid_scale;
    p->kernel = (c.variant == STENCIL_VARIANT_STREAM) ? stencil::stream_kernel_name(p->geo, c.depth)
                                                      : "stencil_generic_kernel";
}

}  // namespace

extern "C" {

const char *stencil_status_str(stencil_status s)
{
    switch (s) {
    case STENCIL_OK: return "STENCIL_OK";
    case STENCIL_ERR_INVALID_ARG: return "STENCIL_ERR_INVALID_ARG";
    case STENCIL_ERR_UNSUPPORTED: return "STENCIL_ERR_UNSUPPORTED";
    case STENCIL_ERR_MISMATCH: return "STENCIL_ERR_MISMATCH";
    case STENCIL_ERR_ALIAS: return "STENCIL_ERR_ALIAS";
    case STENCIL_ERR_NO_MEMORY: return "STENCIL_ERR_NO_MEMORY";
    case STENCIL_ERR_HIP: return "STENCIL_ERR_HIP";
    }
    return "unknown status";
}

const char *stencil_last_error(void)
{
    return g_last_error.c_str();
}

int32_t stencil_num_points(int32_t shape, int32_t ndim, int32_t radius)
{
    return points(shape, ndim, radius);
}

stencil_status stencil_plan(const stencil_desc *desc, stencil_plan_t *out_plan)
{
    if (out_plan == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    Geometry g{};
    stencil_status st = validate_desc(desc, &g);
    if (st != STENCIL_OK)
        return st;

    int variant = desc->variant;
    const bool stream_ok = stencil::stream_supported(g);
    if (variant == STENCIL_VARIANT_AUTO)
        variant = stream_ok ? STENCIL_VARIANT_STREAM : STENCIL_VARIANT_GENERIC;
    if (variant == STENCIL_VARIANT_STREAM && !stream_ok)
        return fail(STENCIL_ERR_UNSUPPORTED,
                    "no streaming kernel runs this description (they cover the 3D 3x3x3 box, "
                    "2D boxes and 2D/3D stars up to radius 4, a coefficient field only with "
                    "the 3D box, and need an x extent they can tile in 16-byte vectors)");
    const int max_depth = (variant == STENCIL_VARIANT_STREAM) ? stencil::stream_max_depth(g) : 1;
    const int dflt = (variant == STENCIL_VARIANT_STREAM) ? stencil::stream_default_depth(g) : 1;
    int depth = desc->temporal_depth == 0 ? dflt : desc->temporal_depth;
    if (depth > max_depth)
        return fail(STENCIL_ERR_UNSUPPORTED, "temporal_depth %d exceeds %d for this variant",
                    desc->temporal_depth, max_depth);
    if (desc->tile != 0 && !(variant == STENCIL_VARIANT_STREAM && stencil::stream_has_tiles(g)))
        return fail(STENCIL_ERR_UNSUPPORTED, "tile %d: this kernel family has a single tile",
                    desc->tile);

    Plan *p = new (std::nothrow) Plan();
    if (p == nullptr)
        return fail(STENCIL_ERR_NO_MEMORY, "plan allocation failed");
    p->desc = *desc;
    p->geo = g;
    p->variant = variant;
    p->depth = depth;
    p->kernel = (variant == STENCIL_VARIANT_STREAM) ? stencil::stream_kernel_name(g, depth)
                                                    : "stencil_generic_kernel";
    p->scratch_bytes = size_t(g.batch) * size_t(g.vol) * g.elt;
    *out_plan = reinterpret_cast<stencil_plan_t>(p);
    g_last_error.clear();
    return STENCIL_OK;
}

stencil_status stencil_plan_query(stencil_plan_t plan, stencil_plan_info *info)
{
    if (plan == nullptr || info == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "plan or info is NULL");
    const Plan *p = reinterpret_cast<const Plan *>(plan);
    info->variant = p->variant;
    info->temporal_depth = p->depth;
    info->scratch_bytes = int64_t(p->scratch_bytes);
    info->kernel = p->kernel;
    // the plan's tile; 0 resolved to the default where the plan runs a one-step kernel
    // with two tiles
    const int resolved =
        p->variant == STENCIL_VARIANT_STREAM ? stencil::stream_tile(p->geo, p->depth) : 0;
    info->tile = resolved != 0 ? resolved : p->geo.tile;
    info->grid_scale = p->geo.grid_scale;
    return STENCIL_OK;
}

stencil_status stencil_destroy(stencil_plan_t plan)
{
    if (plan == nullptr)
        return STENCIL_OK;
    Plan *p = reinterpret_cast<Plan *>(plan);
    stencil_status st = STENCIL_OK;
    if (p->device >= 0) {
        int cur = -1;
        if (hipGetDevice(&cur) == hipSuccess && cur != p->device)
            (void)hipSetDevice(p->device);
        if (p->stage_done && hipEventSynchronize(p->stage_done) != hipSuccess)
            st = STENCIL_ERR_HIP;
        if (p->stage_done)
            (void)hipEventDestroy(p->stage_done);
        if (p->h_stage)
            (void)hipHostFree(p->h_stage);
        if (p->d_coeff)
            (void)hipFree(p->d_coeff);
        if (p->scratch)
            (void)hipFree(p->scratch);
        if (cur >= 0 && cur != p->device)
            (void)hipSetDevice(cur);
    }
    delete p;
    if (st != STENCIL_OK)
        return fail(st, "event synchronisation failed while destroying the plan");
    return STENCIL_OK;
}

stencil_status stencil_apply(stencil_plan_t plan, const void *in, void *out,
                             const int64_t dims[3], const void *coeffs,
                             const void *coeff_field, int32_t radius, int32_t boundary,
                             int32_t steps, hipStream_t stream)
{
    // ---- host-only validation ------------------------------------------------------
    if (plan == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "plan is NULL");
    Plan *p = reinterpret_cast<Plan *>(plan);
    const Geometry &g = p->geo;
    stencil_status st =
        check_call(p, in, out, dims, coeffs, coeff_field, radius, boundary, steps);
    if (st != STENCIL_OK)
        return st;
    const bool fast = stencil::runs_fast(p, in, out, coeff_field);
    const int launches = stencil::launch_count(p, fast, steps);

    // ---- device state (first use) --------------------------------------------------
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (p->device >= 0 && dev != p->device)
        return fail(STENCIL_ERR_MISMATCH, "plan belongs to device %d, current device is %d",
                    p->device, dev);
    p->device = dev;
    const size_t wbytes = size_t(g.channels) * size_t(g.npts) * g.elt;
    // each resource is created on its own, so that a call after a failed first use
    // completes the set instead of running with part of it missing
    if (p->d_coeff == nullptr) {
        if ((e = hipMalloc(&p->d_coeff, wbytes)) != hipSuccess) {
            p->d_coeff = nullptr;
            return fail(STENCIL_ERR_NO_MEMORY, "hipMalloc(%zu) for weights: %s", wbytes,
                        hipGetErrorString(e));
        }
        p->coeff_valid = false;
    }
    if (p->h_stage == nullptr) {
        if ((e = hipHostMalloc(&p->h_stage, wbytes, hipHostMallocDefault)) != hipSuccess) {
            p->h_stage = nullptr;
            return fail(STENCIL_ERR_NO_MEMORY, "hipHostMalloc(%zu): %s", wbytes,
                        hipGetErrorString(e));
        }
    }
    if (p->stage_done == nullptr) {
        if ((e = hipEventCreateWithFlags(&p->stage_done, hipEventDisableTiming)) != hipSuccess) {
            p->stage_done = nullptr;
            return hip_fail(e, "hipEventCreateWithFlags");
        }
    }
    if (p->h_cache.size() != wbytes)
        p->h_cache.assign(wbytes, 0);
    if (launches > 1 && p->scratch == nullptr) {
        if ((e = hipMalloc(&p->scratch, p->scratch_bytes)) != hipSuccess) {
            p->scratch = nullptr;
            return fail(STENCIL_ERR_NO_MEMORY, "hipMalloc(%zu) for the ping-pong grid: %s",
                        p->scratch_bytes, hipGetErrorString(e));
        }
    }
    // ---- weights: upload only when they changed --------------------------------------
    if (!p->coeff_valid || std::memcmp(p->h_cache.data(), coeffs, wbytes) != 0) {
        if ((e = hipEventSynchronize(p->stage_done)) != hipSuccess)
            return hip_fail(e, "hipEventSynchronize(staging)");
        std::memcpy(p->h_stage, coeffs, wbytes);
        if ((e = hipMemcpyAsync(p->d_coeff, p->h_stage, wbytes, hipMemcpyHostToDevice,
                                stream)) != hipSuccess)
            return hip_fail(e, "hipMemcpyAsync(weights)");
        if ((e = hipEventRecord(p->stage_done, stream)) != hipSuccess)
            return hip_fail(e, "hipEventRecord(staging)");
        std::memcpy(p->h_cache.data(), coeffs, wbytes);
        p->coeff_valid = true;
    }

    // ---- steps ------------------------------------------------------------------------
    return stencil::enqueue_steps(p, fast, in, out, coeff_field, p->d_coeff, p->scratch, steps,
                                  stream);
}

stencil_status stencil_tune(stencil_plan_t plan, const void *in, void *out,
                            const int64_t dims[3], const void *coeffs, const void *coeff_field,
                            int32_t steps, double tolerance, int32_t reps, hipStream_t stream,
                            stencil_tune_report *report)
{
    // ---- host-only validation (as stencil_apply, plus the tuning arguments) ----------
    if (plan == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "plan is NULL");
    Plan *p = reinterpret_cast<Plan *>(plan);
    const Geometry &g = p->geo;
    stencil_status st =
        check_call(p, in, out, dims, coeffs, coeff_field, g.radius, g.boundary, steps);
    if (st != STENCIL_OK)
        return st;
    if (steps < 1)
        return fail(STENCIL_ERR_INVALID_ARG, "tuning needs steps >= 1 (got %d)", steps);
    if (reps < 0 || reps > 1000)
        return fail(STENCIL_ERR_INVALID_ARG, "reps must be in 0..1000 (got %d)", reps);
    if (tolerance != tolerance)
        return fail(STENCIL_ERR_INVALID_ARG, "tolerance is NaN");
    if (reps == 0)
        reps = 5;
    if (report != nullptr) {
        std::memset(report, 0, sizeof *report);
        report->chosen = -1;
    }

    // ---- candidates: the reference first --------------------------------------------
    Config cands[STENCIL_TUNE_MAX_CANDIDATES];
    int nc = 0;
    cands[nc++] = {STENCIL_VARIANT_GENERIC, 1, 0, 0};
    const bool aligned = aligned16(in) && aligned16(out) &&
                         (coeff_field == nullptr || aligned16(coeff_field));
    if (aligned && stencil::stream_supported(g)) {
        int depths[4];
        const int nd = stencil::stream_tune_depths(g, depths);
        for (int di = 0; di < nd; ++di) {
            const int depth = depths[di];
            const bool tiles = depth == 1 && stencil::stream_has_tiles(g);
            for (int tile = tiles ? 1 : 0; tile <= (tiles ? 2 : 0); ++tile)
                for (int scale = -1; scale <= 2; ++scale)
                    if (nc < STENCIL_TUNE_MAX_CANDIDATES)
                        cands[nc++] = {STENCIL_VARIANT_STREAM, depth, tile, scale};
        }
    }

    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (p->device >= 0 && dev != p->device)
        return fail(STENCIL_ERR_MISMATCH, "plan belongs to device %d, current device is %d",
                    p->device, dev);

    const Config saved = config_of(p);
    const int64_t n = g.batch * g.vol;
    const size_t bytes = size_t(n) * g.elt;
    void *ref = nullptr;
    double *part = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    auto release = [&]() {
        if (e0)
            (void)hipEventDestroy(e0);
        if (e1)
            (void)hipEventDestroy(e1);
        if (ref)
            (void)hipFree(ref);
        if (part)
            (void)hipFree(part);
    };
    auto abort_with = [&](stencil_status s2) {
        (void)hipStreamSynchronize(stream);
        set_config(p, saved);
        release();
        return s2;
    };
    if ((e = hipMalloc(&ref, bytes)) != hipSuccess) {
        ref = nullptr;
        return abort_with(fail(e == hipErrorOutOfMemory ? STENCIL_ERR_NO_MEMORY : STENCIL_ERR_HIP,
                               "hipMalloc(%zu) for the reference: %s", bytes,
                               hipGetErrorString(e)));
    }
    if ((e = hipMalloc(&part, stencil::kCheckPartials * sizeof(double))) != hipSuccess) {
        part = nullptr;
        return abort_with(fail(e == hipErrorOutOfMemory ? STENCIL_ERR_NO_MEMORY : STENCIL_ERR_HIP,
                               "hipMalloc for the check: %s", hipGetErrorString(e)));
    }
    if ((e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess)
        return abort_with(hip_fail(e, "hipEventCreate"));
    // max |a - b| (or max |a|) on the GPU, read back after the stream drains
    auto max_abs = [&](const void *a, const void *b, double *result) -> stencil_status {
        hipError_t e2 = stencil::launch_max_abs(g.dtype, a, b, n, part, stream);
        if (e2 != hipSuccess)
            return hip_fail(e2, "max-abs check launch");
        if ((e2 = hipMemcpyAsync(result, part, sizeof(double), hipMemcpyDeviceToHost, stream)) !=
                hipSuccess ||
            (e2 = hipStreamSynchronize(stream)) != hipSuccess)
            return hip_fail(e2, "max-abs check read-back");
        return STENCIL_OK;
    };
    auto run = [&](const Config &c, void *dst) {
        set_config(p, c);
        return stencil_apply(plan, in, dst, dims, coeffs, coeff_field, g.radius, g.boundary,
                             steps, stream);
    };

    // ---- reference and tolerance ---------------------------------------------------------
    if ((st = run(cands[0], ref)) != STENCIL_OK)
        return abort_with(st);
    double tol = tolerance;
    if (tol < 0) {
        double in_max = 0.0;
        if ((st = max_abs(in, nullptr, &in_max)) != STENCIL_OK)
            return abort_with(st);
        const double c = (g.dtype == STENCIL_F32) ? 2e-5 : 2e-12;
        tol = c * double(steps) * (in_max > 1.0 ? in_max : 1.0);  // NaN input: NaN, no pass
    }

    // ---- every candidate through the validity gate --------------------------------------
    bool valid[STENCIL_TUNE_MAX_CANDIDATES] = {};
    double errs[STENCIL_TUNE_MAX_CANDIDATES] = {};
    double ms[STENCIL_TUNE_MAX_CANDIDATES];
    int last = -1;
    for (int i = 0; i < nc; ++i) {
        if ((st = run(cands[i], out)) != STENCIL_OK)
            return abort_with(st);
        last = i;
        if ((st = max_abs(out, ref, &errs[i])) != STENCIL_OK)
            return abort_with(st);
        valid[i] = errs[i] <= tol;  // false for NaN
        ms[i] = -1.0;
    }

    // ---- timing: kTuneRounds interleaved rounds over the valid candidates; a candidate's
    // time is the mean of `reps` calls in its fastest round, so that a clock or cache
    // transient during one candidate's turn does not decide the choice
    constexpr int kTuneRounds = 3;
    for (int round = 0; round < kTuneRounds; ++round) {
        for (int i = 0; i < nc; ++i) {
            if (!valid[i])
                continue;
            if ((e = hipEventRecord(e0, stream)) != hipSuccess)
                return abort_with(hip_fail(e, "hipEventRecord"));
            for (int r = 0; r < reps; ++r)
                if ((st = run(cands[i], out)) != STENCIL_OK)
                    return abort_with(st);
            last = i;
            float total = 0.f;
            if ((e = hipEventRecord(e1, stream)) != hipSuccess ||
                (e = hipEventSynchronize(e1)) != hipSuccess ||
                (e = hipEventElapsedTime(&total, e0, e1)) != hipSuccess)
                return abort_with(hip_fail(e, "timing events"));
            const double t = double(total) / reps;
            if (ms[i] < 0 || t < ms[i])
                ms[i] = t;
        }
    }
    int best = -1;
    for (int i = 0; i < nc; ++i)
        if (valid[i] && (best < 0 || ms[i] < ms[best]))
            best = i;
    if (report != nullptr) {
        for (int i = 0; i < nc; ++i) {
            stencil_tune_entry &r = report->entry[i];
            r.variant = cands[i].variant;
            r.temporal_depth = cands[i].depth;
            r.tile = cands[i].tile;
            r.grid_scale = cands[i].grid_scale;
            r.valid = valid[i] ? 1 : 0;
            r.max_abs_err = errs[i];
            r.ms = ms[i];
        }
        report->count = nc;
    }
    if (report != nullptr)
        report->tolerance = tol;
    if (best < 0)
        return abort_with(fail(STENCIL_ERR_UNSUPPORTED,
                               "no candidate stayed within tolerance %g of the reference", tol));

    // ---- fix the winner; leave its result in `out` --------------------------------------
    if (best != last && (st = run(cands[best], out)) != STENCIL_OK)
        return abort_with(st);
    set_config(p, cands[best]);
    if ((e = hipStreamSynchronize(stream)) != hipSuccess)
        return abort_with(hip_fail(e, "hipStreamSynchronize"));
    release();
    if (report != nullptr)
        report->chosen = best;
    g_last_error.clear();
    return STENCIL_OK;
}

}  // extern "C"
