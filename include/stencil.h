/*
 * stencil.h -- C ABI of the MI355X (gfx950) structured-grid stencil library.
 *
 * The operator is the one of the HIERA scientific-computing case study (experimental
 * setup, paragraph "Case-study protocol"): a box stencil of radius R applied as a
 * zero-padded cross-correlation with padding R and stride 1, repeated step after step on
 * its own output, with per-step latency as the figure of merit.  This library computes
 * that operator and its generalisations on one GPU:
 *
 *   one step   u_{t+1}[p] = k[p] * sum_{j} w_c[j] * u_t(p + O[j])      (k = 1 without field)
 *   u_t(q)     = 0 outside the grid            (STENCIL_ZERO, re-applied at every step)
 *              = u_t[q mod dims]               (STENCIL_PERIODIC, non-negative modulo)
 *   result     = u_steps, written to `out`;   steps = 0 copies `in` to `out`.
 *
 * It is a cross-correlation: no flip of the weights (weight j multiplies u(p + O[j])).
 * The coefficient field k, when present, is indexed by the OUTPUT point p.
 *
 * Layout.  Row-major (C order).  3D extents dims = {nz, ny, nx}, 2D dims = {ny, nx, -}; the
 * last axis is unit-stride.  `batch` independent volumes are stored back to back (conv
 * layout N x C x D x H x W gives batch = N * C); volume b uses weight set c = b % channels.
 *
 * Offset order O[j] (the order of each weight set):
 *   STENCIL_BOX : lexicographic over (oz, oy, ox) in [-R, R]^3 (2D: (oy, ox)), ox fastest,
 *                 i.e. a correlation kernel W[oz+R][oy+R][ox+R] flattened in C order;
 *   STENCIL_STAR: the centre first, then for each axis from slowest to fastest the
 *                 offsets -R..-1, +1..+R along that axis (1 + 2*ndim*R points).
 *
 * Arithmetic.  f32 grids are computed in fp32, f64 grids in fp64; the summation order
 * and fused multiply-adds are the kernel's choice (results agree with an fp64 evaluation
 * to within rounding).
 *
 * Errors.  Every call returns a stencil_status and never aborts.  All argument checks are
 * made on the host before any HIP call, so invalid calls fail the same way on a machine
 * without a GPU.  HIP failures return STENCIL_ERR_HIP.  A human-readable detail of the
 * last failure on the calling thread is returned by stencil_last_error().
 */
#ifndef MI355X_STENCIL_H
#define MI355X_STENCIL_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct stencil_plan_s *stencil_plan_t; /* opaque; created and freed by the library */

typedef enum {
    STENCIL_OK = 0,
    STENCIL_ERR_INVALID_ARG = 1, /* NULL pointer, bad enum, non-positive extent, steps < 0 */
    STENCIL_ERR_UNSUPPORTED = 2, /* radius or shape beyond the supported range, or a forced
                                    variant that cannot run this description */
    STENCIL_ERR_MISMATCH = 3,    /* apply() arguments disagree with the plan */
    STENCIL_ERR_ALIAS = 4,       /* out overlaps in or the coefficient field */
    STENCIL_ERR_NO_MEMORY = 5,   /* host or device allocation failed */
    STENCIL_ERR_HIP = 6          /* a HIP runtime call failed (detail in stencil_last_error) */
} stencil_status;

typedef enum { STENCIL_F32 = 0, STENCIL_F64 = 1 } stencil_dtype;
typedef enum { STENCIL_STAR = 0, STENCIL_BOX = 1 } stencil_shape;
typedef enum { STENCIL_ZERO = 0, STENCIL_PERIODIC = 1 } stencil_boundary;

/* Kernel families.  AUTO lets the planner choose; the others force one (for testing and
 * tuning) and make stencil_plan() fail with STENCIL_ERR_UNSUPPORTED where it cannot run. */
typedef enum {
    STENCIL_VARIANT_AUTO = 0,
    STENCIL_VARIANT_GENERIC = 1, /* one thread per point, any description */
    STENCIL_VARIANT_STREAM = 2   /* tiled kernels: 3D 3x3x3 box and 2D/3D stars up to radius
                                    4, 2.5D z-streaming in 3D; x extent a multiple of 16
                                    bytes (box: whole 64-lane row segments) */
} stencil_variant;

typedef struct {
    int32_t ndim;            /* 2 or 3 */
    int64_t dims[3];         /* slowest..fastest extents, each >= 1; 2D uses dims[0..1] */
    int64_t batch;           /* number of contiguous volumes, >= 1 */
    int32_t channels;        /* number of weight sets, >= 1; volume b uses set b % channels */
    int32_t dtype;           /* stencil_dtype */
    int32_t shape;           /* stencil_shape */
    int32_t radius;          /* STAR: 0..4; BOX: 0..4 in 2D, 0..3 in 3D */
    int32_t boundary;        /* stencil_boundary */
    int32_t has_coeff_field; /* 1: out[p] = k[p] * sum_j w[j] * u(p + O[j]); 0: no field */
    int32_t variant;         /* stencil_variant; 0 = AUTO */
    int32_t temporal_depth;  /* steps fused per launch where the variant supports it;
                                0 = planner's choice, 1 = one launch per step.  The
                                streaming variant fuses up to 2 steps for 2D boxes and 3D
                                stars, up to 4 for fp32 and 3 for fp64 radius-1 3D stars;
                                a larger value is STENCIL_ERR_UNSUPPORTED.  A call whose step count is not
                                a multiple ends with a shallower pass */
    int32_t tile;            /* workgroup tile of the one-step streaming kernels that have
                                two: 0 = planner's choice, 1 = the smaller, 2 = the larger
                                (3D star: 32- or 64-row x-y tiles; 3D box: 4 or 8 rows per
                                lane).  The fused two-step kernels have one tile and ignore
                                it.  Non-zero with a kernel family that has one tile, or with
                                the generic variant: STENCIL_ERR_UNSUPPORTED */
    int32_t grid_scale;      /* number of workgroups relative to the planner's choice, as a
                                power of two, -2..2 (0 = planner's choice).  The streaming
                                kernels split their streaming axis into correspondingly more
                                or fewer chunks; the generic kernel caps its grid
                                accordingly.  Results do not depend on it */
} stencil_desc;

typedef struct {
    int32_t variant;         /* the stencil_variant chosen (never AUTO) */
    int32_t temporal_depth;  /* steps fused per launch */
    int64_t scratch_bytes;   /* device bytes the plan allocates for steps > 1 */
    const char *kernel;      /* base name of the dominant GPU kernel (static string) */
    int32_t tile;            /* the description's tile; where the plan's kernel is a
                                one-step kernel with two tiles and the description says 0,
                                the tile the planner resolved it to (1 or 2) */
    int32_t grid_scale;      /* workgroup-count exponent in use */
} stencil_plan_info;

/* One candidate of stencil_tune(): a (variant, temporal depth, tile, grid scale) point. */
typedef struct {
    int32_t variant;         /* STENCIL_VARIANT_GENERIC or STENCIL_VARIANT_STREAM */
    int32_t temporal_depth;
    int32_t tile;
    int32_t grid_scale;
    int32_t valid;           /* 1: max_abs_err <= the tolerance (NaN is never valid) */
    int32_t reserved;
    double max_abs_err;      /* max over all points of |candidate - reference| */
    double ms;               /* mean time of one call of `steps` steps in the fastest of
                                the timing rounds; -1 if not timed (invalid) */
} stencil_tune_entry;

#define STENCIL_TUNE_MAX_CANDIDATES 20

typedef struct {
    int32_t count;           /* candidates tried (entries filled) */
    int32_t chosen;          /* index of the candidate fixed in the plan; -1 if none */
    double tolerance;        /* the tolerance applied */
    stencil_tune_entry entry[STENCIL_TUNE_MAX_CANDIDATES];
} stencil_tune_report;

/*
 * stencil_plan -- validate a description and create a plan for it.
 *   desc      : host pointer, read during the call only.
 *   out_plan  : receives the plan; set to NULL on failure.
 * No HIP call is made here: device memory (coefficients, and the ping-pong grid used when
 * steps > 1) is allocated by the first stencil_apply() that needs it, on the device current
 * at that time, and the plan stays tied to that device.
 * Returns STENCIL_OK, INVALID_ARG, UNSUPPORTED or NO_MEMORY.
 */
stencil_status stencil_plan(const stencil_desc *desc, stencil_plan_t *out_plan);

/*
 * stencil_apply -- run `steps` steps of the planned operator on `stream`.
 * (Operator: HIERA, "Case-study protocol"; generalisations as described at the top.)
 *   plan        : from stencil_plan().
 *   in          : device pointer, batch volumes of dims (dtype of the plan); read only.
 *   out         : device pointer, same size; receives u_steps.  Must not overlap `in`.
 *   dims        : host array {nz, ny, nx} (2D: {ny, nx, ignored}); must equal the plan's.
 *   coeffs      : host pointer, channels * npoints weights of the plan's dtype, in the
 *                 offset order above; copied before the call returns.
 *   coeff_field : device pointer to one dims-shaped field per volume (same layout as `in`),
 *                 or NULL; must be non-NULL exactly when the plan has a field.
 *   radius, boundary : must equal the plan's (re-stated so a call reads as the operator).
 *   steps       : >= 0.
 *   stream      : HIP stream (NULL = default stream); all work is enqueued on it.
 * Ownership: in, out and coeff_field belong to the caller and must stay valid until the
 * stream work completes.  Asynchronous: returns once the work is enqueued.  Calls on one
 * plan must be ordered on one stream at a time (the plan's ping-pong grid and coefficient
 * buffer are reused), and one plan must not be called from several host threads at once;
 * different plans may be used concurrently.  Pointers or x extents that do not meet a
 * fast kernel's alignment select a slower kernel; they are not an error.
 * Returns STENCIL_OK, INVALID_ARG, MISMATCH, ALIAS, NO_MEMORY or ERR_HIP.
 */
stencil_status stencil_apply(stencil_plan_t plan, const void *in, void *out,
                             const int64_t dims[3], const void *coeffs,
                             const void *coeff_field, int32_t radius, int32_t boundary,
                             int32_t steps, hipStream_t stream);

/*
 * stencil_tune -- empirical plan-time search with a validity gate.  It mirrors the
 * objective of HIERA (Sec. "Problem Formulation and Framework Overview", Eq. 2): the
 * fastest candidate among those explored, subject to Valid(x) = 1.  Here the candidates
 * are launch configurations of this library's kernels on the caller's own buffers.
 *   Reference: the generic kernel (one thread per point, one launch per step) applied to
 *     `in` for `steps` steps.
 *   Candidates (at most STENCIL_TUNE_MAX_CANDIDATES): the generic kernel itself; then,
 *     when the streaming variant can run the description and `in`, `out` and
 *     `coeff_field` are 16-byte aligned, the temporal depths 1, 2 and the deepest the
 *     description supports (3 or 4 for radius-1 3D stars; a depth of 3 is not tried
 *     where 4 is possible) x every tile of the one-step kernels (1, 2, or the single
 *     tile) x grid_scale in {-1, 0, 1, 2} (at most 17 candidates).
 *   Validity: a candidate's `out` must satisfy max_p |out - reference| <= tolerance (on the
 *     GPU, all points).  Invalid candidates are not timed.
 *   Timing: three rounds over the valid candidates (the validity run is each one's
 *     warm-up); in each round, `reps` calls between HIP events on `stream`.  A
 *     candidate's time is the mean call time of its fastest round.
 *   Result: the fastest valid candidate is fixed in the plan (variant, depth, tile,
 *     grid_scale; stencil_plan_query reports it), and `out` holds its result, i.e. `out`
 *     receives u_steps exactly as stencil_apply() would.
 * Arguments are those of stencil_apply() (same checks, same ownership), plus:
 *   steps     : >= 1.
 *   tolerance : < 0 selects c * steps * max(1, max|in|) with c = 2e-5 (f32) or 2e-12 (f64),
 *               twice the per-step bound the library's tests hold each kernel to against
 *               an fp64 evaluation; 0 accepts only results identical to the reference; a
 *               positive value is an absolute bound.  Plans with a coefficient field whose
 *               values exceed 1 in magnitude should pass their own bound.
 *   reps      : timed calls per candidate, 1..1000 (0 selects 5).
 *   report    : host pointer filled with every candidate, or NULL.
 * Synchronous: returns after the stream has drained.  It allocates one grid-sized device
 * buffer for the reference (freed before returning) and uses the plan's buffers.
 * Returns STENCIL_OK, INVALID_ARG, MISMATCH, ALIAS, NO_MEMORY, UNSUPPORTED (no candidate
 * passed the gate; the plan is left unchanged) or ERR_HIP.
 */
stencil_status stencil_tune(stencil_plan_t plan, const void *in, void *out,
                            const int64_t dims[3], const void *coeffs, const void *coeff_field,
                            int32_t steps, double tolerance, int32_t reps, hipStream_t stream,
                            stencil_tune_report *report);

/* Sizes of the device scratch stencil_apply_noalloc() uses: one static array per GPU,
 * held until the process ends. */
#define STENCIL_NOALLOC_WEIGHT_BYTES (64 * 1024)        /* channels * npoints weights */
#define STENCIL_NOALLOC_GRID_BYTES (64 * 1024 * 1024)   /* intermediate grid of a call */

/*
 * stencil_apply_noalloc -- stencil_apply for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, and harnesses that forbid hipMalloc.
 * It calls no hipMalloc, hipFree or other allocating routine, and it does not use or
 * create the plan's device buffers.  It runs the same kernels in the same launch
 * configuration as stencil_apply, so its results are identical.
 *   Arguments, ownership and checks: those of stencil_apply().
 *   Scratch: the weights and, for a call of more than one launch, the intermediate grid
 *     live in a static device array of STENCIL_NOALLOC_WEIGHT_BYTES +
 *     STENCIL_NOALLOC_GRID_BYTES bytes per GPU, created with the library's code object
 *     and looked up on the first call on each device.  Nothing in it needs clearing: each
 *     call's weights are in place before its first launch -- uploaded with hipMemcpyAsync
 *     on `stream` (staged before the call returns), or left as they are when the device's
 *     weight region already holds the same bytes from an earlier call (the library keeps
 *     a host copy of what it last uploaded per device, in static memory).  Under stream
 *     capture, one call with the same weights before the capture leaves no copy in the
 *     captured work.
 *   Limits: channels * npoints * sizeof(dtype) <= STENCIL_NOALLOC_WEIGHT_BYTES, and, when
 *     the call makes more than one launch (steps beyond the plan's temporal depth, or
 *     more than one step on the generic kernel), batch * volume * sizeof(dtype) <=
 *     STENCIL_NOALLOC_GRID_BYTES; otherwise STENCIL_ERR_UNSUPPORTED, before any HIP call.
 *   Concurrency: every call on a GPU shares that GPU's scratch.  Calls ordered on one
 *     stream are safe; calls that overlap in time on one GPU (other streams, other
 *     threads) race on it and must not be issued.
 * Returns STENCIL_OK, INVALID_ARG, MISMATCH, ALIAS, UNSUPPORTED or ERR_HIP.
 */
stencil_status stencil_apply_noalloc(stencil_plan_t plan, const void *in, void *out,
                                     const int64_t dims[3], const void *coeffs,
                                     const void *coeff_field, int32_t radius, int32_t boundary,
                                     int32_t steps, hipStream_t stream);

/*
 * stencil_destroy -- free a plan and its device memory.  NULL is accepted.  The caller
 * must make sure no enqueued work still uses the plan (synchronise its stream first).
 */
stencil_status stencil_destroy(stencil_plan_t plan);

/* Describe the plan's choices.  info: host pointer.  Returns OK or INVALID_ARG. */
stencil_status stencil_plan_query(stencil_plan_t plan, stencil_plan_info *info);

/* Number of offsets: STAR 1 + 2*ndim*R, BOX (2R+1)^ndim; -1 for an invalid description. */
int32_t stencil_num_points(int32_t shape, int32_t ndim, int32_t radius);

/* Static name of a status code ("STENCIL_OK", ...); "unknown status" otherwise. */
const char *stencil_status_str(stencil_status status);

/* Detail of the last failure on the calling thread ("" if none).  Valid until the next
 * call on that thread. */
const char *stencil_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MI355X_STENCIL_H */
