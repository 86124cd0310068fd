// fg_host.hpp — host-side helpers shared by the library's C entry points:
// the per-thread error text and HIP launch-status mapping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include <tuple>
#include <utility>

#include "fgemm.h"

namespace fg {

// Records a formatted description of the failure for fg_last_error() on
// this thread and returns `st`.
fg_status fail(fg_status st, const char* fmt, ...);
// Clears the recorded description (called at the start of each entry point).
void clear_error();
// Enqueues `kernel` and returns the status of this launch alone (not an
// error some earlier, unrelated HIP call left pending on the thread). The
// arguments are converted to the kernel's parameter types first.
template <class... P, size_t... I>
hipError_t launch_packed(void (*kernel)(P...), dim3 grid, dim3 block, size_t shmem, hipStream_t s,
                         std::tuple<P...>& args, std::index_sequence<I...>) {
  void* ptrs[sizeof...(P) + 1] = {static_cast<void*>(&std::get<I>(args))..., nullptr};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, s);
}
// Launch trace (fg_trace_begin): the slot this launch records its events
// into (its "before" event is recorded here), or −1 when no trace is open on
// the thread or the trace is full; trace_launch_end records the "after"
// event and the kernel.
int trace_launch_begin(hipStream_t s);
void trace_launch_end(int slot, hipStream_t s, const void* kernel);

template <class... P, class... A>
hipError_t launch(void (*kernel)(P...), dim3 grid, dim3 block, size_t shmem, hipStream_t s, A&&... args) {
  static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
  std::tuple<P...> packed(static_cast<P>(std::forward<A>(args))...);
  const int slot = trace_launch_begin(s);
  const hipError_t e = launch_packed(kernel, grid, block, shmem, s, packed, std::index_sequence_for<P...>{});
  if (slot >= 0) trace_launch_end(slot, s, reinterpret_cast<const void*>(kernel));
  return e;
}

// Collects the launch statuses of one entry point: the first failure wins.
struct Launches {
  hipError_t first = hipSuccess;
  void add(hipError_t e) {
    if (first == hipSuccess) first = e;
  }
};
// Maps the statuses of the launches this call made to an fg_status. On a
// failure the runtime's pending error (this call's own) is consumed, so it
// is not reported again to the next unrelated HIP user on the thread.
fg_status check_launch(const char* what, const Launches& l);

// Run epochs for the arrival words of K-split exchanges: distinct for every
// launch of the process (0 is skipped), so a word left by any other launch
// never matches.
unsigned next_epoch();

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace fg
