// swr_internal.h -- host functions shared between the C ABI's source files.
// Not part of the public ABI.
#pragma once

#include <stdint.h>

#include "../../include/swr.h"

namespace swr {

// Returns the device address of the library's static scratch array on the
// device that runs `stream` (NULL: the current device), or NULL when the HIP
// runtime fails.
typedef void* (*ScratchFn)(void* stream);

// The exact forward (the body of swr_exact_forward).  With scratch == NULL
// the workspace is the caller's `workspace`; otherwise `workspace` is ignored
// and the launches use the array that scratch(stream) returns, which holds
// scratch_bytes bytes: a problem needing more is rejected with
// SWR_ERR_SCRATCH.  Every argument is validated before scratch() or any
// other HIP runtime call.
int exact_forward_impl(const swr_problem_t* p, const void* x, const void* a, const void* b, const void* c,
                       const float* h0, void* y, float* carriers, float* h_last, void* workspace,
                       ScratchFn scratch, int64_t scratch_bytes, void* stream);

}  // namespace swr
