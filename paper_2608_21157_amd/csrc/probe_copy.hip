// probe_copy.hip -- 16-byte streaming copy: the achievable read+write HBM ceiling, and
// the reference for scaling hardware byte counters.
//
// Each workgroup copies one contiguous chunk, four 16-byte vectors per thread in flight,
// with non-temporal loads and stores (the fastest plain copy measured on MI355X:
// ~5.5 TB/s read+write, against ~5.0 TB/s for a cached grid-stride copy).
#include <hip/hip_runtime.h>

#include "stencil_probe.h"

namespace {

typedef float V4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 4;
constexpr long long kBlocks = 16384;

__global__ __launch_bounds__(256) void stencil_probe_copy_kernel(const V4 *__restrict__ src,
                                                                 V4 *__restrict__ dst,
                                                                 long long n, long long chunk)
{
    const long long beg = (long long)blockIdx.x * chunk;
    const long long end = beg + chunk < n ? beg + chunk : n;
    for (long long i = beg + threadIdx.x; i < end; i += 256 * kUnroll) {
        V4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long j = i + u * 256;
            if (j < end)
                v[u] = __builtin_nontemporal_load(src + j);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long j = i + u * 256;
            if (j < end)
                __builtin_nontemporal_store(v[u], dst + j);
        }
    }
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
    if (blocks > kBlocks)
        blocks = kBlocks;
    const long long chunk = (n + blocks - 1) / blocks;
    blocks = (n + chunk - 1) / chunk;
    stencil_probe_copy_kernel<<<dim3(unsigned(blocks)), dim3(256), 0, stream>>>(
        static_cast<const V4 *>(src), static_cast<V4 *>(dst), n, chunk);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
