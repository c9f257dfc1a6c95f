// Internal entry points shared between the host planner (fno_plan.cpp) and
// the allocation-free entry point (fno_noalloc.hip).  Not part of the ABI.
#pragma once

#include "fno_spectral_conv.h"

namespace fno {

// The forward call behind fno_spectral_conv_fwd.  With build_plan false the
// descriptor's plan must already exist on the current device
// (FNO_ERR_INVALID_ARGUMENT otherwise), the workspace is checked against the
// cached plan, and no device memory is allocated and no event created.
fno_status fwd_impl(const fno_conv_desc* d, const void* x, const fno_weights* w, void* y,
                    void* x_hat_out, void* ws, size_t ws_len, hipStream_t s, bool build_plan);

}  // namespace fno
