// Error reporting shared by the C ABI sources: each failing entry point
// records a message (returned by opscale_last_error) and its status.
#pragma once
#include <hip/hip_runtime.h>

#include "opscale.h"

namespace opscale {

// Records the printf-style message and returns st.
opscale_status fail(opscale_status st, const char* fmt, ...);
// OPSCALE_ERR_HIP with "<what>: <HIP error string>".
opscale_status hip_fail(hipError_t e, const char* what);

}  // namespace opscale
