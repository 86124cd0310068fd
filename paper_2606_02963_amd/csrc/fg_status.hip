// fg_status.hip — status strings, per-thread error text and launch checks.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include <atomic>
#include <vector>

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

static std::atomic<unsigned> g_epoch{0};
unsigned next_epoch() {
  unsigned e;
  do e = g_epoch.fetch_add(1, std::memory_order_relaxed) + 1; while (e == 0);
  return e;
}

fg_status check_launch(const char* what, const Launches& l) {
  if (l.first == hipSuccess) return FG_OK;
  (void)hipGetLastError();
  return fail(FG_ERR_HIP, "%s: kernel launch failed: %s", what, hipGetErrorString(l.first));
}

// The open launch trace of a thread: two events per launch slot, created
// on first use and kept for the thread's later traces.
struct TraceState {
  std::vector<hipEvent_t> ev;
  std::vector<const void*> kernel;
  int cap = 0, n = 0;
  bool open = false;
};
static thread_local TraceState g_trace;

int trace_launch_begin(hipStream_t s) {
  TraceState& t = g_trace;
  if (!t.open || t.n >= t.cap) return -1;
  const int i = t.n++;
  (void)hipEventRecord(t.ev[2 * i], s);
  return i;
}

void trace_launch_end(int slot, hipStream_t s, const void* kernel) {
  g_trace.kernel[slot] = kernel;
  (void)hipEventRecord(g_trace.ev[2 * slot + 1], s);
}

}  // namespace fg

extern "C" fg_status fg_trace_begin(int32_t capacity) {
  using namespace fg;
  clear_error();
  TraceState& t = g_trace;
  if (capacity < 1 || capacity > (1 << 20))
    return fail(FG_ERR_INVALID_ARG, "fg_trace_begin: capacity %d outside 1..2^20", capacity);
  while ((int64_t)t.ev.size() < 2 * (int64_t)capacity) {
    hipEvent_t e;
    const hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) {
      (void)hipGetLastError();
      return fail(FG_ERR_HIP, "fg_trace_begin: hipEventCreate failed: %s", hipGetErrorString(err));
    }
    t.ev.push_back(e);
  }
  t.kernel.assign(capacity, nullptr);
  t.cap = capacity;
  t.n = 0;
  t.open = true;
  return FG_OK;
}

extern "C" int32_t fg_trace_end(void) {
  fg::g_trace.open = false;
  return fg::g_trace.n;
}

extern "C" fg_status fg_trace_read(int32_t i, float* ms, const char** kernel) {
  using namespace fg;
  clear_error();
  TraceState& t = g_trace;
  if (t.open) return fail(FG_ERR_INVALID_ARG, "fg_trace_read: the trace is still open");
  if (i < 0 || i >= t.n) return fail(FG_ERR_INVALID_ARG, "fg_trace_read: launch %d outside 0..%d", i, t.n - 1);
  if (ms != nullptr) {
    hipError_t err = hipEventSynchronize(t.ev[2 * i + 1]);
    if (err == hipSuccess) err = hipEventElapsedTime(ms, t.ev[2 * i], t.ev[2 * i + 1]);
    if (err != hipSuccess) {
      (void)hipGetLastError();
      return fail(FG_ERR_HIP, "fg_trace_read: %s", hipGetErrorString(err));
    }
  }
  if (kernel != nullptr) {
    const char* name = hipKernelNameRefByPtr(t.kernel[i], nullptr);
    *kernel = name != nullptr ? name : "";
  }
  return FG_OK;
}

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
