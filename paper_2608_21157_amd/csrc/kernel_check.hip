// kernel_check.hip -- max |a - b| (or max |a|) over a whole grid, on the GPU: the validity
// gate of the plan-time tuner (a candidate is kept only if its result stays within a
// tolerance of the reference kernel's result at every point).
//
// Two passes: a grid-stride pass writes one maximum per workgroup, then one workgroup
// reduces those.  A NaN anywhere propagates to the result.
#include "plan.hpp"

namespace stencil {
namespace {

constexpr int kThreads = 256;
constexpr int kBlocks = kCheckPartials - 1;  // first-pass workgroups at most

// maximum that keeps a NaN once it has seen one
__device__ __forceinline__ double max_nan(double m, double v)
{
    return (v > m || v != v) ? v : m;
}

__device__ __forceinline__ double block_max(double m)
{
    __shared__ double red[kThreads];
    red[threadIdx.x] = m;
    __syncthreads();
    for (int s = kThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s)
            red[threadIdx.x] = max_nan(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    return red[0];
}

template <typename T>
__global__ __launch_bounds__(kThreads) void stencil_max_abs_kernel(const T *__restrict__ a,
                                                                   const T *__restrict__ b,
                                                                   long long n,
                                                                   double *__restrict__ partial)
{
    double m = 0.0;
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const double d = b ? double(a[i]) - double(b[i]) : double(a[i]);
        m = max_nan(m, fabs(d));
    }
    m = block_max(m);
    if (threadIdx.x == 0)
        partial[1 + blockIdx.x] = m;
}

__global__ __launch_bounds__(kThreads) void stencil_max_abs_final_kernel(double *partial,
                                                                         int count)
{
    double m = 0.0;
    for (int i = threadIdx.x; i < count; i += kThreads)
        m = max_nan(m, partial[1 + i]);
    m = block_max(m);
    if (threadIdx.x == 0)
        partial[0] = m;
}

}  // namespace

hipError_t launch_max_abs(int dtype, const void *a, const void *b, int64_t n, double *partial,
                          hipStream_t stream)
{
    if (n < 1)
        return hipErrorInvalidValue;
    long long blocks = (n + kThreads - 1) / kThreads;
    if (blocks > kBlocks)
        blocks = kBlocks;
    if (dtype == STENCIL_F32)
        stencil_max_abs_kernel<float><<<dim3(blocks), dim3(kThreads), 0, stream>>>(
            static_cast<const float *>(a), static_cast<const float *>(b), n, partial);
    else
        stencil_max_abs_kernel<double><<<dim3(blocks), dim3(kThreads), 0, stream>>>(
            static_cast<const double *>(a), static_cast<const double *>(b), n, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    stencil_max_abs_final_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(partial, int(blocks));
    return hipGetLastError();
}

}  // namespace stencil
