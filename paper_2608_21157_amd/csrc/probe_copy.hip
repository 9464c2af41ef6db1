// probe_copy.hip -- plain 16-byte streaming copy (HBM ceiling and counter calibration).
#include <hip/hip_runtime.h>

#include "stencil_probe.h"

namespace {

__global__ __launch_bounds__(256) void stencil_probe_copy_kernel(const float4 *__restrict__ src,
                                                                 float4 *__restrict__ dst,
                                                                 long long n)
{
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

}  // namespace

extern "C" int stencil_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t stream)
{
    if (src == nullptr || dst == nullptr || bytes < 0 || bytes % 16 != 0 ||
        (reinterpret_cast<uintptr_t>(src) & 15u) || (reinterpret_cast<uintptr_t>(dst) & 15u))
        return 1;
    const long long n = bytes / 16;
    if (n == 0)
        return 0;
    long long blocks = (n + 255) / 256;
    if (blocks > 256 * 32)
        blocks = 256 * 32;  // 32 workgroups per CU, grid-stride beyond that
    stencil_probe_copy_kernel<<<dim3(unsigned(blocks)), dim3(256), 0, stream>>>(
        static_cast<const float4 *>(src), static_cast<float4 *>(dst), n);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
