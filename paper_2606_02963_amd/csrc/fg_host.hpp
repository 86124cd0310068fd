// fg_host.hpp — host-side helpers shared by the library's C entry points:
// the per-thread error text and HIP launch-status mapping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include "fgemm.h"

namespace fg {

// Records a formatted description of the failure for fg_last_error() on
// this thread and returns `st`.
fg_status fail(fg_status st, const char* fmt, ...);
// Clears the recorded description (called at the start of each entry point).
void clear_error();
// Maps the launch status of the kernels just enqueued to an fg_status.
fg_status check_launch(const char* what);

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace fg
