// noalloc.hip -- stencil_apply_noalloc: the apply call for callers that cannot allocate
// device memory (code under graph capture, tight serving loops, harnesses that forbid
// hipMalloc).
//
// It runs the same kernels, in the same launch configuration, as stencil_apply.  The
// device memory stencil_apply keeps in the plan -- the weight buffer and the ping-pong
// grid of a call of more than one launch -- comes instead from `scratch`, one static
// device array per GPU that lives as long as the process.  The first call on a device
// looks up that device's address of the array (hipGetSymbolAddress, with the device
// current) and keeps it; every later call uses that address, never the array's name,
// which in host code is only a stand-in for the symbol.
//
// Nothing in `scratch` must start at zero: a call's weights are in place before its first
// launch (uploaded, unless the region already holds the same bytes), and the first launch
// that reads the intermediate grid reads what the launch before it wrote.  Every call on
// a GPU shares that GPU's array, so calls that overlap in time on one GPU (on different
// streams, or from different threads without ordering) race on it; calls ordered on one
// stream do not.
#include <cstring>
#include <mutex>

#include "entry.hpp"
#include "plan.hpp"

namespace {

constexpr size_t kWeightBytes = STENCIL_NOALLOC_WEIGHT_BYTES;
constexpr size_t kGridBytes = STENCIL_NOALLOC_GRID_BYTES;
constexpr int kMaxDevices = 64;

}  // namespace

// the weights at offset 0, the intermediate grid at kWeightBytes (a multiple of 256)
static __device__ __align__(256) unsigned char scratch[kWeightBytes + kGridBytes];

namespace {

static_assert(kWeightBytes % 256 == 0, "the grid region must stay 256-byte aligned");

std::mutex g_scratch_mutex;
unsigned char *g_scratch_ptr[kMaxDevices] = {};
// the bytes last uploaded into each device's weight region (static host memory), so that
// a call whose weights are already there skips the upload
unsigned char g_weights_host[kMaxDevices][kWeightBytes];
size_t g_weights_len[kMaxDevices] = {};

// This device's address of `scratch`, looked up once per device (the device is current).
stencil_status device_scratch(int dev, unsigned char **out)
{
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return stencil::hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (ptr == nullptr)
            return stencil::fail(STENCIL_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL");
        g_scratch_ptr[dev] = static_cast<unsigned char *>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return STENCIL_OK;
}

}  // namespace

extern "C" stencil_status stencil_apply_noalloc(stencil_plan_t plan, const void *in, void *out,
                                                const int64_t dims[3], const void *coeffs,
                                                const void *coeff_field, int32_t radius,
                                                int32_t boundary, int32_t steps,
                                                hipStream_t stream)
{
    using stencil::fail;
    // ---- host-only validation, the same as stencil_apply's, plus the scratch limits ----
    if (plan == nullptr)
        return fail(STENCIL_ERR_INVALID_ARG, "plan is NULL");
    const stencil::Plan *p = reinterpret_cast<const stencil::Plan *>(plan);
    const stencil::Geometry &g = p->geo;
    stencil_status st =
        stencil::check_call(p, in, out, dims, coeffs, coeff_field, radius, boundary, steps);
    if (st != STENCIL_OK)
        return st;
    const size_t wbytes = size_t(g.channels) * size_t(g.npts) * g.elt;
    if (wbytes > kWeightBytes)
        return fail(STENCIL_ERR_UNSUPPORTED,
                    "the weights take %zu bytes; the no-alloc scratch holds %zu", wbytes,
                    kWeightBytes);
    const bool fast = stencil::runs_fast(p, in, out, coeff_field);
    const int launches = stencil::launch_count(p, fast, steps);
    const size_t grid_bytes = size_t(g.batch) * size_t(g.vol) * g.elt;
    if (launches > 1 && grid_bytes > kGridBytes)
        return fail(STENCIL_ERR_UNSUPPORTED,
                    "a call of %d launches needs a %zu-byte intermediate grid; the no-alloc "
                    "scratch holds %zu (calls of one launch have no such limit)",
                    launches, grid_bytes, kGridBytes);

    // ---- this device's scratch ---------------------------------------------------------
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return stencil::hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(STENCIL_ERR_UNSUPPORTED, "device %d beyond the %d the library tracks", dev,
                    kMaxDevices);
    unsigned char *base = nullptr;
    if ((st = device_scratch(dev, &base)) != STENCIL_OK)
        return st;

    // ---- weights, then the launches ----------------------------------------------------
    // The weights are uploaded unless the device's weight region already holds these
    // bytes (from any plan's earlier call: all calls on a device share the region).  The
    // upload is ordered on `stream` before the launches; a copy from pageable host memory
    // is staged by the runtime before it returns, so `coeffs` may be reused as soon as
    // this call returns.  A call that skips the upload relies on the earlier call being
    // ordered before it, which the concurrency rule above already requires.
    if (steps > 0) {
        std::lock_guard<std::mutex> lock(g_scratch_mutex);
        if (g_weights_len[dev] != wbytes ||
            std::memcmp(g_weights_host[dev], coeffs, wbytes) != 0) {
            g_weights_len[dev] = 0;  // unknown contents until the copy is enqueued
            if ((e = hipMemcpyAsync(base, coeffs, wbytes, hipMemcpyHostToDevice, stream)) !=
                hipSuccess)
                return stencil::hip_fail(e, "hipMemcpyAsync(weights into the scratch)");
            std::memcpy(g_weights_host[dev], coeffs, wbytes);
            g_weights_len[dev] = wbytes;
        }
    }
    return stencil::enqueue_steps(p, fast, in, out, coeff_field, base, base + kWeightBytes,
                                  steps, stream);
}
