// entry.hpp -- host helpers shared by the C entry points (abi.cpp, noalloc.hip): error
// recording, argument checks and the step loop of an apply call.
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

#include "plan.hpp"
#include "stencil.h"

namespace stencil {

// Failure helpers of the entry points: record a detail for stencil_last_error() and
// return the status (printf-style), or clear the detail after a successful call.
stencil_status fail(stencil_status st, const char *fmt, ...);
stencil_status hip_fail(hipError_t e, const char *what);
void clear_error();

// Host-side argument checks of an apply call against its plan (no HIP call).
stencil_status check_call(const Plan *p, const void *in, const void *out, const int64_t dims[3],
                          const void *coeffs, const void *coeff_field, int32_t radius,
                          int32_t boundary, int32_t steps);

// Whether a call runs the plan's streaming kernels (16-byte aligned pointers), and how
// many launches a call of `steps` steps then makes.
bool runs_fast(const Plan *p, const void *in, const void *out, const void *coeff_field);
int launch_count(const Plan *p, bool fast, int steps);

// Enqueue a call's launches on `stream`: `w` holds the weights on the device, `grid` is
// the intermediate grid of a call of more than one launch (batch * volume elements; not
// read when the call makes one launch).  steps = 0 copies `in` to `out`.
stencil_status enqueue_steps(const Plan *p, bool fast, const void *in, void *out,
                             const void *coeff_field, const void *w, void *grid, int steps,
                             hipStream_t stream);

}  // namespace stencil
