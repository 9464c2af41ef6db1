// kernel_stream.hip -- dispatch of the tiled kernel families (3x3x3 box, radius-R star).
#include "plan.hpp"

namespace stencil {

bool stream_supported(const Geometry &g)
{
    return box_stream_supported(g) || star_stream_supported(g);
}

int stream_max_depth(const Geometry &g)
{
    return 1;
}

const char *stream_kernel_name(const Geometry &g)
{
    if (box_stream_supported(g))
        return "stencil_box3_stream_kernel";
    if (star_stream_supported(g))
        return "stencil_star_stream_kernel";
    return "";
}

hipError_t launch_stream(const Geometry &g, const void *src, void *dst, const void *field,
                         const void *w, int depth, hipStream_t stream)
{
    if (depth != 1)
        return hipErrorInvalidValue;
    if (box_stream_supported(g))
        return launch_box_stream(g, src, dst, field, w, stream);
    if (star_stream_supported(g))
        return launch_star_stream(g, src, dst, w, stream);
    return hipErrorInvalidValue;
}

}  // namespace stencil
