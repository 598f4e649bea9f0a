// Host-side argument checks shared between the C ABI's source files.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "ssn.h"

namespace ssn {

// Validation of ssn_reparam_backward's arguments (shapes, NULLs, alignment,
// overlaps); check_ws: also the caller's workspace pointer and size.
ssn_status_t reparam_backward_args(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k,
                                   const void* H, const void* Zp, const void* U, const void* G,
                                   const float* GT, const void* GH, const float* GZp,
                                   const void* workspace, size_t workspace_bytes, bool check_ws);

}  // namespace ssn
