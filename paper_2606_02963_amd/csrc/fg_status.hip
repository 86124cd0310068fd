// fg_status.hip — status strings, per-thread error text and launch checks.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include "fg_host.hpp"
#include "fgemm.h"

namespace fg {

static thread_local char g_last_error[512];

fg_status fail(fg_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

void clear_error() { g_last_error[0] = '\0'; }

fg_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(FG_ERR_HIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
  return FG_OK;
}

}  // namespace fg

extern "C" const char* fg_status_str(fg_status s) {
  switch (s) {
    case FG_OK: return "FG_OK: success";
    case FG_ERR_INVALID_ARG: return "FG_ERR_INVALID_ARG: invalid argument";
    case FG_ERR_UNSUPPORTED: return "FG_ERR_UNSUPPORTED: no kernel for this request";
    case FG_ERR_ALIGNMENT: return "FG_ERR_ALIGNMENT: pointer or dimension misaligned";
    case FG_ERR_WORKSPACE: return "FG_ERR_WORKSPACE: workspace missing or too small";
    case FG_ERR_HIP: return "FG_ERR_HIP: HIP runtime error";
  }
  return "unknown fg_status";
}

extern "C" const char* fg_last_error(void) { return fg::g_last_error; }
