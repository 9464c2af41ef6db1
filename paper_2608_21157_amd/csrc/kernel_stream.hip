// kernel_stream.hip -- 2.5D z-streaming kernels (placeholder until the tiled kernels land).
#include "plan.hpp"

namespace stencil {

bool stream_supported(const Geometry &) { return false; }
int stream_max_depth(const Geometry &) { return 1; }
const char *stream_kernel_name(const Geometry &) { return ""; }
hipError_t launch_stream(const Geometry &, const void *, void *, const void *, const void *,
                         int, hipStream_t)
{
    return hipErrorInvalidValue;
}

}  // namespace stencil
