/*
 * A plain C99 consumer of the library's C ABI (include/stencil.h): built with gcc and run
 * by tests/test_c_consumer.py.  It exercises only calls that fail or succeed on the host
 * (point counts, status strings, plan validation, plan queries, argument checks of
 * stencil_apply that reject the call before any HIP call), so it runs the same with or
 * without a GPU.  Exit status 0 when every check holds; each failure is printed.
 */
#include <stdio.h>
#include <string.h>

#include "stencil.h"

static int failures = 0;

static void expect(int ok, const char *what)
{
    if (!ok) {
        printf("FAIL: %s (last error: %s)\n", what, stencil_last_error());
        ++failures;
    }
}

static stencil_desc headline(void)
{
    stencil_desc d;
    memset(&d, 0, sizeof d);
    d.ndim = 3;
    d.dims[0] = 512;
    d.dims[1] = 512;
    d.dims[2] = 512;
    d.batch = 1;
    d.channels = 1;
    d.dtype = STENCIL_F32;
    d.shape = STENCIL_STAR;
    d.radius = 4;
    d.boundary = STENCIL_ZERO;
    return d;
}

int main(void)
{
    /* point counts: star 1 + 2 ndim R, box (2R + 1)^ndim */
    expect(stencil_num_points(STENCIL_STAR, 3, 4) == 25, "3D star R=4 has 25 points");
    expect(stencil_num_points(STENCIL_STAR, 2, 1) == 5, "2D star R=1 has 5 points");
    expect(stencil_num_points(STENCIL_BOX, 3, 1) == 27, "3D box R=1 has 27 points");
    expect(stencil_num_points(STENCIL_BOX, 2, 3) == 49, "2D box R=3 has 49 points");
    expect(stencil_num_points(STENCIL_BOX, 4, 1) == -1, "ndim 4 is invalid");
    expect(strcmp(stencil_status_str(STENCIL_ERR_ALIAS), "STENCIL_ERR_ALIAS") == 0,
           "status string");

    /* plan validation */
    stencil_plan_t p = NULL;
    stencil_desc d = headline();
    d.ndim = 1;
    expect(stencil_plan(&d, &p) == STENCIL_ERR_INVALID_ARG && p == NULL, "ndim 1 rejected");
    d = headline();
    d.radius = 5;
    expect(stencil_plan(&d, &p) == STENCIL_ERR_UNSUPPORTED, "star radius 5 unsupported");
    d = headline();
    d.shape = STENCIL_BOX;
    d.radius = 4;
    expect(stencil_plan(&d, &p) == STENCIL_ERR_UNSUPPORTED, "3D box radius 4 unsupported");
    expect(stencil_plan(NULL, &p) == STENCIL_ERR_INVALID_ARG, "NULL desc rejected");

    /* a valid plan and its query */
    d = headline();
    expect(stencil_plan(&d, &p) == STENCIL_OK && p != NULL, "headline plan");
    stencil_plan_info info;
    memset(&info, 0, sizeof info);
    expect(stencil_plan_query(p, &info) == STENCIL_OK, "plan query");
    expect(info.variant == STENCIL_VARIANT_STREAM && info.temporal_depth == 2 &&
               info.kernel != NULL && strcmp(info.kernel, "stencil_star_tb2_kernel") == 0,
           "the headline plan fuses two steps in the star kernel");

    /* stencil_apply argument checks (all rejected before any HIP call) */
    float w[25] = {0};
    const int64_t dims[3] = {512, 512, 512};
    const int64_t wrong[3] = {512, 512, 256};
    void *a = (void *)(size_t)0x100000, *b = (void *)(size_t)0x40100000;
    expect(stencil_apply(p, NULL, b, dims, w, NULL, 4, STENCIL_ZERO, 4, NULL) ==
               STENCIL_ERR_INVALID_ARG, "NULL input rejected");
    expect(stencil_apply(p, a, b, wrong, w, NULL, 4, STENCIL_ZERO, 4, NULL) ==
               STENCIL_ERR_MISMATCH, "dims that differ from the plan");
    expect(stencil_apply(p, a, b, dims, w, NULL, 3, STENCIL_ZERO, 4, NULL) ==
               STENCIL_ERR_MISMATCH, "radius that differs from the plan");
    expect(stencil_apply(p, a, b, dims, w, NULL, 4, STENCIL_PERIODIC, 4, NULL) ==
               STENCIL_ERR_MISMATCH, "boundary that differs from the plan");
    expect(stencil_apply(p, a, b, dims, w, a, 4, STENCIL_ZERO, 4, NULL) ==
               STENCIL_ERR_MISMATCH, "field given to a plan without one");
    expect(stencil_apply(p, a, (char *)a + 64, dims, w, NULL, 4, STENCIL_ZERO, 4, NULL) ==
               STENCIL_ERR_ALIAS, "overlapping in and out");
    expect(stencil_apply(p, a, b, dims, w, NULL, 4, STENCIL_ZERO, -1, NULL) ==
               STENCIL_ERR_INVALID_ARG, "negative steps");
    expect(strlen(stencil_last_error()) > 0, "a failure leaves a detail string");

    expect(stencil_destroy(p) == STENCIL_OK, "destroy");
    expect(stencil_destroy(NULL) == STENCIL_OK, "destroy NULL");

    if (failures == 0)
        printf("c consumer: all checks passed\n");
    return failures == 0 ? 0 : 1;
}
