// kernel_stream.hip -- dispatch of the tiled kernel families (3x3x3 box, radius-R star).
#include "plan.hpp"

namespace stencil {

bool stream_supported(const Geometry &g)
{
    return box_stream_supported(g) || box2_stream_supported(g) || box2_tb2_supported(g) ||
           star_stream_supported(g);
}

int stream_max_depth(const Geometry &g)
{
    if (star_tbs_supported(g))
        return star_tbs_max_depth(g);
    return (star_tb2_supported(g) || box2_tb2_supported(g)) ? 2 : 1;
}

int stream_tune_depths(const Geometry &g, int *depths)
{
    // 1, 2 and the deepest: three steps per pass is never the fastest where four are
    // possible (measured on fp32 radius 1, 256^3 and 512^3), so the tuner skips it there
    int n = 0;
    depths[n++] = 1;
    const int dmax = stream_max_depth(g);
    if (dmax >= 2)
        depths[n++] = 2;
    if (dmax >= 3)
        depths[n++] = dmax;
    return n;
}

int stream_default_depth(const Geometry &g)
{
    // Fusing two steps halves HBM traffic but costs redundant stage-1 work on the halo
    // bands and LDS traffic that grow with the radius.  Measured on MI355X, 4 steps per
    // call, zero boundary, Gpoints/s at one step per launch -> two fused steps:
    //   fp32 512^3:      R=1 643 -> 1205, R=2 617 -> 1005, R=3 598 -> 792, R=4 594 -> 699
    //   fp64 256x512^2:  R=1 332 -> 631,  R=2 301 -> 500,  R=3 307 -> 387, R=4 311 -> 338
    // 2D boxes: two steps per pass measured 1.26x faster per step (10240^2 fp64, radius 3)
    // radius 1 with a working set beyond the Infinity Cache: four steps per pass in fp32,
    // three in fp64 (kernel_star_tbs.hip; fp32 512^3, 10 steps: 1235 -> 1406-1471
    // Gpoints/s; fp64 512^3, 9 steps: 507 -> 770-784); inside it two (fp32 256^3, 10
    // steps: 1300 against 1230 with four)
    if (star_tbs_supported(g) && streaming_stores(g))
        return star_tbs_max_depth(g);
    if (box2_tb2_supported(g) || star_tb2_supported(g))
        return 2;
    return 1;
}

bool stream_has_tiles(const Geometry &g)
{
    // box3: 4 or 8 rows per lane; star (one step): 32- or 64-row workgroup tiles
    return box_stream_supported(g) || star_stream_supported(g);
}

int stream_tile(const Geometry &g, int depth)
{
    if (depth != 1 || !stream_has_tiles(g))
        return 0;
    if (g.tile != 0)
        return g.tile;
    // defaults, measured on MI355X: the 3D box runs 8 rows per lane (tile 2) without a
    // coefficient field and 4 (tile 1) with one (interleaved rounds, Gpoints/s, tile 1 ->
    // 2: depthwise 8x32x128^3 fp32 701 -> 707, 2x32x128^3 fp64 347 -> 353; 512^3 with a
    // field 510 -> 503); the star runs 64 x 64 tiles in 3D (tile 2) and 64 x 32 tiles in
    // 2D (tile 1)
    if (box_stream_supported(g))
        return g.field ? 1 : 2;
    return g.ndim == 3 ? 2 : 1;
}

const char *stream_kernel_name(const Geometry &g, int depth)
{
    if (box_stream_supported(g))
        return "stencil_box3_stream_kernel";
    if (box2_tb2_supported(g) && depth == 2)
        return "stencil_box2_tb2_kernel";
    if (box2_stream_supported(g))
        return "stencil_box2_stream_kernel";
    if (star_tbs_supported(g) && depth >= 3)
        return "stencil_star_tbs_kernel";
    if (star_tb2_supported(g) && depth == 2)
        return "stencil_star_tb2_kernel";
    if (star_stream_supported(g))
        return "stencil_star_stream_kernel";
    return "";
}

hipError_t launch_stream(const Geometry &g, const void *src, void *dst, const void *field,
                         const void *w, int depth, hipStream_t stream)
{
    if (depth >= 3 && star_tbs_supported(g))
        return launch_star_tbs(g, src, dst, w, depth, stream);
    if (depth == 2 && star_tb2_supported(g))
        return launch_star_tb2(g, src, dst, w, stream);
    if (depth == 2 && box2_tb2_supported(g))
        return launch_box2_stream(g, src, dst, w, 2, stream);
    if (depth != 1)
        return hipErrorInvalidValue;
    if (box_stream_supported(g))
        return launch_box_stream(g, src, dst, field, w, stream);
    if (box2_stream_supported(g))
        return launch_box2_stream(g, src, dst, w, 1, stream);
    if (star_stream_supported(g))
        return launch_star_stream(g, src, dst, w, stream);
    return hipErrorInvalidValue;
}

}  // namespace stencil
