// plan.hpp -- internal plan state and kernel launchers of the stencil library.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include <hip/hip_runtime.h>

#include "stencil.h"

namespace stencil {

// Geometry of one apply: every extent is the 3D view (nz = 1 for a 2D grid).
struct Geometry {
    int ndim;
    int64_t nz, ny, nx;
    int64_t vol;      // nz * ny * nx
    int64_t batch;
    int channels;
    int npts;
    int shape;        // STENCIL_STAR / STENCIL_BOX
    int radius;
    int boundary;     // STENCIL_ZERO / STENCIL_PERIODIC
    bool field;
    int dtype;        // STENCIL_F32 / STENCIL_F64
    size_t elt;       // bytes per element
    int tile;         // one-step streaming tile: 0 = default, 1 = smaller, 2 = larger
    int grid_scale;   // workgroup count relative to the default, as a power of two
};

// A kernel's default workgroup (or wavefront) count scaled by 2^grid_scale, at least 1.
inline long long scaled_target(long long dflt, int grid_scale)
{
    long long t = grid_scale >= 0 ? dflt << grid_scale : dflt >> -grid_scale;
    return t < 1 ? 1 : t;
}

// Workgroups of `kernel` the current device runs at once: resident blocks per CU (from
// the kernel's registers and LDS, through the HIP occupancy API) times the CU count; 256
// if the query fails.  Launchers call it once per kernel (a function-local static): every
// device the library drives is taken to be the same model.
template <typename K>
int resident_blocks(K kernel, int threads)
{
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) !=
            hipSuccess ||
        cus < 1 || per_cu < 1)
        return 256;
    return cus * per_cu;
}

struct Plan {
    stencil_desc desc{};
    Geometry geo{};                // geo.tile and geo.grid_scale hold the launch choice
    int variant = STENCIL_VARIANT_GENERIC;
    int depth = 1;                 // steps fused per launch
    const char *kernel = "";

    int device = -1;               // device of the first apply
    void *d_coeff = nullptr;       // channels * npts weights (device)
    void *h_stage = nullptr;       // pinned staging of the weights
    hipEvent_t stage_done = nullptr;
    std::vector<unsigned char> h_cache;  // weights last uploaded
    bool coeff_valid = false;
    void *scratch = nullptr;       // ping-pong grid for steps > 1
    size_t scratch_bytes = 0;
};

// Whether output stores should bypass the caches.  Streaming (non-temporal) stores raise
// read+write HBM throughput, but a working set that fits the 256 MB Infinity Cache (in,
// out and the ping-pong grid of a multi-step call) is better kept there.
inline bool streaming_stores(const Geometry &g)
{
    const double grid = double(g.batch) * double(g.vol) * double(g.elt);
    const double footprint = grid * (g.field ? 4.0 : 3.0);
    return footprint > 192.0 * 1024 * 1024;
}

// Launch one pass of `depth` steps (depth <= plan.depth) from src to dst.  `w` is the
// device weight buffer (channels * npts of the plan's dtype).
hipError_t launch_generic(const Geometry &g, const void *src, void *dst, const void *field,
                          const void *w, hipStream_t stream);

// Kernel families behind the streaming variant.
bool box_stream_supported(const Geometry &g);
hipError_t launch_box_stream(const Geometry &g, const void *src, void *dst, const void *field,
                             const void *w, hipStream_t stream);

bool star_stream_supported(const Geometry &g);
hipError_t launch_star_stream(const Geometry &g, const void *src, void *dst, const void *w,
                              hipStream_t stream);

bool box2_stream_supported(const Geometry &g);
bool box2_tb2_supported(const Geometry &g);
hipError_t launch_box2_stream(const Geometry &g, const void *src, void *dst, const void *w,
                              int depth, hipStream_t stream);

// Two star steps fused in one pass (3D).
bool star_tb2_supported(const Geometry &g);
hipError_t launch_star_tb2(const Geometry &g, const void *src, void *dst, const void *w,
                           hipStream_t stream);

// Three or four star steps fused in one pass (3D, radius 1; four in fp32, three in fp64).
bool star_tbs_supported(const Geometry &g);
int star_tbs_max_depth(const Geometry &g);
hipError_t launch_star_tbs(const Geometry &g, const void *src, void *dst, const void *w,
                           int depth, hipStream_t stream);

// Temporal depths stencil_tune tries for this geometry (ascending, at most 4 entries);
// returns their number.
int stream_tune_depths(const Geometry &g, int *depths);

// Whether the one-step streaming kernel of this geometry offers two tiles (tile 1 / 2).
bool stream_has_tiles(const Geometry &g);

// The tile a streaming launch of `depth` steps runs: for a one-step kernel with two tiles,
// the plan's tile or, for 0, the family default (1 or 2); 0 for kernels with one tile.
// The launchers and stencil_plan_query both use it.
int stream_tile(const Geometry &g, int depth);

// max |a - b| over n elements of the given dtype (max |a| when b is NULL), computed on the
// GPU.  `partial` is device memory for kCheckPartials doubles; the result lands in
// partial[0] (NaN if any difference is NaN).
constexpr int kCheckPartials = 1025;
hipError_t launch_max_abs(int dtype, const void *a, const void *b, int64_t n, double *partial,
                          hipStream_t stream);

// 2.5D z-streaming kernels.  `supported` says whether the kernel family can run a
// geometry (shape, radius, alignment of the x extent); launch_* run one pass.
bool stream_supported(const Geometry &g);
int stream_max_depth(const Geometry &g);
int stream_default_depth(const Geometry &g);
const char *stream_kernel_name(const Geometry &g, int depth);
hipError_t launch_stream(const Geometry &g, const void *src, void *dst, const void *field,
                         const void *w, int depth, hipStream_t stream);

}  // namespace stencil
