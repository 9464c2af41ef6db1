// kernel_generic.hip -- one thread per output point, any offset set, radius and extent.
//
// One step of the operator (HIERA, "Case-study protocol": zero-padded cross-correlation,
// stride 1; generalised to star/box offsets, periodic wrap, an output-indexed field and
// batched volumes).  This kernel is the fallback for descriptions the streaming kernels do
// not tile (2D grids, tiny or odd extents, misaligned pointers) and the first-parity path.
// Offsets are recomputed from the offset index instead of read from a table.
#include "plan.hpp"

namespace stencil {
namespace {

struct GenericParams {
    int64_t nz, ny, nx, vol, total;
    int npts, shape, ndim, radius, channels;
};

// Offset j of the documented weight order.
__device__ __forceinline__ void offset_of(const GenericParams &p, int j, int &oz, int &oy,
                                          int &ox)
{
    const int R = p.radius;
    if (p.shape == STENCIL_BOX) {
        const int side = 2 * R + 1;
        ox = j % side - R;
        const int t = j / side;
        oy = t % side - R;
        oz = (p.ndim == 3) ? t / side - R : 0;
    } else {
        oz = oy = ox = 0;
        if (j == 0)
            return;
        const int k = j - 1;
        const int axis = k / (2 * R) + (p.ndim == 3 ? 0 : 1);
        const int r = k % (2 * R);
        const int o = (r < R) ? r - R : r - R + 1;
        if (axis == 0)
            oz = o;
        else if (axis == 1)
            oy = o;
        else
            ox = o;
    }
}

template <bool PERIODIC>
__device__ __forceinline__ bool resolve(int64_t &q, int64_t n)
{
    if (q >= 0 && q < n)
        return true;
    if (!PERIODIC)
        return false;
    q %= n;
    if (q < 0)
        q += n;
    return true;
}

template <typename T, bool PERIODIC, bool FIELD>
__global__ __launch_bounds__(256) void stencil_generic_kernel(
    const T *__restrict__ in, T *__restrict__ out, const T *__restrict__ field,
    const T *__restrict__ w, GenericParams p)
{
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < p.total; i += stride) {
        const int64_t b = i / p.vol;
        const int64_t r = i - b * p.vol;
        const int64_t x = r % p.nx;
        const int64_t y = (r / p.nx) % p.ny;
        const int64_t z = r / (p.nx * p.ny);
        const T *src = in + b * p.vol;
        const T *wb = w + (b % p.channels) * p.npts;
        T acc = T(0);
        for (int j = 0; j < p.npts; ++j) {
            int oz, oy, ox;
            offset_of(p, j, oz, oy, ox);
            int64_t qz = z + oz, qy = y + oy, qx = x + ox;
            if (resolve<PERIODIC>(qz, p.nz) && resolve<PERIODIC>(qy, p.ny) &&
                resolve<PERIODIC>(qx, p.nx))
                acc = fma(wb[j], src[(qz * p.ny + qy) * p.nx + qx], acc);
        }
        if (FIELD)
            acc *= field[i];
        out[i] = acc;
    }
}

template <typename T>
hipError_t launch_t(const Geometry &g, const void *src, void *dst, const void *field,
                    const void *w, hipStream_t stream)
{
    GenericParams p{g.nz, g.ny, g.nx, g.vol, g.batch * g.vol, g.npts, g.shape, g.ndim,
                    g.radius, g.channels};
    const int threads = 256;
    int64_t blocks = (p.total + threads - 1) / threads;
    const int64_t cap = scaled_target(65536, g.grid_scale);  // grid-stride beyond the cap
    if (blocks > cap)
        blocks = cap;
    const T *s = static_cast<const T *>(src);
    T *d = static_cast<T *>(dst);
    const T *k = static_cast<const T *>(field);
    const T *wt = static_cast<const T *>(w);
    const bool per = g.boundary == STENCIL_PERIODIC;
    if (per && g.field)
        stencil_generic_kernel<T, true, true><<<blocks, threads, 0, stream>>>(s, d, k, wt, p);
    else if (per)
        stencil_generic_kernel<T, true, false><<<blocks, threads, 0, stream>>>(s, d, k, wt, p);
    else if (g.field)
        stencil_generic_kernel<T, false, true><<<blocks, threads, 0, stream>>>(s, d, k, wt, p);
    else
        stencil_generic_kernel<T, false, false><<<blocks, threads, 0, stream>>>(s, d, k, wt, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_generic(const Geometry &g, const void *src, void *dst, const void *field,
                          const void *w, hipStream_t stream)
{
    if (g.dtype == STENCIL_F32)
        return launch_t<float>(g, src, dst, field, w, stream);
    return launch_t<double>(g, src, dst, field, w, stream);
}

}  // namespace stencil
