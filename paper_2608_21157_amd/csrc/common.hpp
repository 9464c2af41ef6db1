// common.hpp -- device helpers shared by the streaming kernels: 16-byte vectors and
// whole-wavefront lane shifts through DPP.
#pragma once

#include <hip/hip_runtime.h>

namespace stencil {

// 16 bytes of T: four floats or two doubles, loaded and stored as one dwordx4 access
// (through the buffer-resource helpers below).
template <typename T>
struct alignas(16) Vec16 {
    static constexpr int N = 16 / sizeof(T);
    T e[N];
};

// DPP controls of the GFX9 family that move data across the whole 64-lane wavefront.
constexpr int kDppWaveShl1 = 0x130;  // lane i reads lane i + 1; lane 63 keeps `old`
constexpr int kDppWaveShr1 = 0x138;  // lane i reads lane i - 1; lane 0 keeps `old`

template <int CTRL>
__device__ __forceinline__ float dpp_move(float src, float old)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src),
                                                      CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ double dpp_move(double src, double old)
{
    const long long s = __double_as_longlong(src), o = __double_as_longlong(old);
    const int lo = __builtin_amdgcn_update_dpp(int(o), int(s), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(int(o >> 32), int(s >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((static_cast<long long>(hi) << 32) |
                                static_cast<unsigned int>(lo));
}

// DPP move whose lanes without a source (lane 0 for wave_shr, lane 63 for wave_shl)
// receive zero (bound_ctrl), so no destination initialisation is needed.
template <int CTRL>
__device__ __forceinline__ float dpp_move_zero(float src)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(src), CTRL, 0xF, 0xF, true));
}

template <int CTRL>
__device__ __forceinline__ double dpp_move_zero(double src)
{
    const long long s = __double_as_longlong(src);
    const int lo = __builtin_amdgcn_mov_dpp(int(s), CTRL, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_mov_dpp(int(s >> 32), CTRL, 0xF, 0xF, true);
    return __longlong_as_double((static_cast<long long>(hi) << 32) |
                                static_cast<unsigned int>(lo));
}

// Value of lane - 1 (lane 0 receives `old`).
template <typename T>
__device__ __forceinline__ T from_left_lane(T v, T old)
{
    return dpp_move<kDppWaveShr1>(v, old);
}

// Value of lane + 1 (lane 63 receives `old`).
template <typename T>
__device__ __forceinline__ T from_right_lane(T v, T old)
{
    return dpp_move<kDppWaveShl1>(v, old);
}

// Value of lane - 1 (lane 0 receives 0) and of lane + 1 (lane 63 receives 0).
template <typename T>
__device__ __forceinline__ T from_left_lane_or_zero(T v)
{
    return dpp_move_zero<kDppWaveShr1>(v);
}

template <typename T>
__device__ __forceinline__ T from_right_lane_or_zero(T v)
{
    return dpp_move_zero<kDppWaveShl1>(v);
}

// Raw buffer access (gfx9 resource word 3 = 0x00020000, stride 0).  Offsets are byte
// offsets from the resource base; a load whose offset is at or beyond num_records returns
// zero and a store there is dropped, which is how out-of-grid rows read the zero padding.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kOutOfRange = 0x7FFFFFF0;  // an offset beyond every resource built here
// cache policy of a buffer access: 0 = default, kNonTemporal = streamed past the caches
// (data read or written once); it measurably raises read+write HBM throughput
constexpr int kNonTemporal = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kBufferWord3);
}

template <typename T, int CP = 0>
__device__ __forceinline__ Vec16<T> bload16(__amdgpu_buffer_rsrc_t r, int off)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CP);
    Vec16<T> out;
    __builtin_memcpy(&out, &v, 16);
    return out;
}

__device__ __forceinline__ float bload1(__amdgpu_buffer_rsrc_t r, int off, float)
{
    return __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

__device__ __forceinline__ double bload1(__amdgpu_buffer_rsrc_t r, int off, double)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
    double d;
    __builtin_memcpy(&d, &v, 8);
    return d;
}

template <typename T, int CP = 0>
__device__ __forceinline__ void bstore16(__amdgpu_buffer_rsrc_t r, int off, const Vec16<T> &v)
{
    __attribute__((ext_vector_type(4))) unsigned int u;
    __builtin_memcpy(&u, &v, 16);
    __builtin_amdgcn_raw_buffer_store_b128(u, r, off, 0, CP);
}

__device__ __forceinline__ int wrap_index(int q, int n)
{
    q %= n;
    return q < 0 ? q + n : q;
}

// Hardware dispatch places workgroup i on XCD (i mod 8).  Renumber so that each XCD
// receives a contiguous range of logical tiles (neighbouring tiles share an L2); blocks
// beyond the largest multiple of 8 keep their index.
__device__ __forceinline__ int xcd_logical_block(int hw_block, int nblocks)
{
    constexpr int kXcds = 8;
    const int per = nblocks / kXcds;
    if (hw_block >= per * kXcds)
        return hw_block;
    return (hw_block % kXcds) * per + hw_block / kXcds;
}

}  // namespace stencil
