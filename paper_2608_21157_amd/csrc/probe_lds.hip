// probe_lds.hip -- LDS access-pattern probe.  Each lane of every wave reads or writes 16
// bytes at a byte offset given per lane (the same 64 offsets for every wave), eight times
// per iteration; the eight accesses add multiples of 4 KiB to the offset, which keeps
// each lane on its banks.  One launch holds one pattern, so the SQ counters of a launch
// (instructions, bank-conflict cycles, LDS-active cycles) describe that pattern alone.
// The patterns measured are those of the fused star kernel's LDS planes and of the
// alternative layouts considered for them.
#include <hip/hip_runtime.h>

#include "stencil_probe.h"

namespace {

typedef float V4 __attribute__((ext_vector_type(4)));

constexpr int kLdsVectors = 4096;   // 64 KiB

struct LaneOffsets {
    int byte[64];
};

__global__ __launch_bounds__(256) void stencil_probe_lds_read_kernel(LaneOffsets t, int iters,
                                                                     float *__restrict__ sink)
{
    __shared__ V4 buf[kLdsVectors];
    for (int i = threadIdx.x; i < kLdsVectors; i += 256)
        buf[i] = V4{float(i), 0.f, 0.f, 0.f};
    __syncthreads();
    const int v0 = t.byte[threadIdx.x & 63] >> 4;
    float acc = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const V4 v = buf[(v0 + u * 256) & (kLdsVectors - 1)];
            acc += v.x + v.y + v.z + v.w;
        }
    }
    if (acc == -1.f)   // never true: keeps the reads
        sink[0] = acc;
}

__global__ __launch_bounds__(256) void stencil_probe_lds_write_kernel(LaneOffsets t, int iters,
                                                                      float *__restrict__ sink)
{
    __shared__ V4 buf[kLdsVectors];
    const int v0 = t.byte[threadIdx.x & 63] >> 4;
    V4 val = V4{float(threadIdx.x), 1.f, 2.f, 3.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
            buf[(v0 + u * 256) & (kLdsVectors - 1)] = val;
        val.x += 1.f;
        // an empty statement that may read memory: the stores of every iteration are kept
        asm volatile("" ::: "memory");
    }
    __syncthreads();
    if (buf[threadIdx.x].x == -1.f)   // never true
        sink[0] = 1.f;
}

}  // namespace

extern "C" int stencil_probe_lds(const int32_t *lane_bytes, int32_t write, int32_t iters,
                                 int32_t blocks, float *sink, hipStream_t stream)
{
    if (lane_bytes == nullptr || sink == nullptr || (write != 0 && write != 1) || iters < 1 ||
        iters > (1 << 20) || blocks < 1 || blocks > (1 << 20))
        return 1;
    LaneOffsets t;
    for (int i = 0; i < 64; ++i) {
        if (lane_bytes[i] < 0 || lane_bytes[i] > 16 * (kLdsVectors - 1) || lane_bytes[i] % 16)
            return 1;
        t.byte[i] = lane_bytes[i];
    }
    if (write)
        stencil_probe_lds_write_kernel<<<dim3(blocks), dim3(256), 0, stream>>>(t, iters, sink);
    else
        stencil_probe_lds_read_kernel<<<dim3(blocks), dim3(256), 0, stream>>>(t, iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
