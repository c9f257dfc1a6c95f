// Internal entry points shared between the host planner (fno_plan.cpp), the
// allocation-free entry point (fno_noalloc.hip) and the block epilogue
// (fno_block.hip).  Not part of the ABI.
#pragma once

#include "fno_spectral_conv.h"

namespace fno {

// The forward call behind fno_spectral_conv_fwd.  With build_plan false the
// descriptor's plan must already exist on the current device
// (FNO_ERR_INVALID_ARGUMENT otherwise), the workspace is checked against the
// cached plan, and no device memory is allocated and no event created.
fno_status fwd_impl(const fno_conv_desc* d, const void* x, const fno_weights* w, void* y,
                    void* x_hat_out, void* ws, size_t ws_len, hipStream_t s, bool build_plan);

// Records a HIP failure as the thread's last error (fno_last_error) and
// returns FNO_ERR_HIP.
fno_status report_hip_error(hipError_t e, const char* what);

// Runs launch(ctx) bracketed by profiling events (fno_profile_enable) under
// the kernel name `name`.
hipError_t timed_launch(const char* name, hipStream_t s, hipError_t (*launch)(void*), void* ctx);

}  // namespace fno
