// moe_noalloc.hip — the MoE step for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops): the same
// launches as moe_grouped_ffn, with the workspace taken from a static device
// array of this file instead of the caller.
//
// Each GPU the library runs on holds its own copy of `scratch` (64 MiB)
// until the process ends. The array's device address is looked up once per
// device with hipGetSymbolAddress and kept; the host-side name of the array
// is never passed to a kernel or a copy. Every call on a device uses that
// device's one array, so calls that overlap in time on one GPU (different
// streams or threads) race on it: the caller serialises them. Nothing in the
// MoE step's workspace must start at zero (the routing launch writes every
// per-block expert count, the placement writes the whole m-tile prefix, and
// h and the slot outputs are written before they are read), so the array is
// never cleared and whatever a previous call left in it is overwritten.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "fg_host.hpp"
#include "fg_moe.hpp"
#include "fgemm.h"

namespace fg {

constexpr size_t MOE_SCRATCH_BYTES = (size_t)64 << 20;
constexpr int MAX_DEVICES = 64;

static __device__ __attribute__((aligned(256))) char scratch[MOE_SCRATCH_BYTES];

static std::atomic<void*> g_scratch[MAX_DEVICES];
static std::mutex g_scratch_mu;

// Device address of the current device's copy of `scratch`.
static fg_status scratch_on_device(const char* fn, void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(FG_ERR_HIP, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
  }
  if (dev < 0 || dev >= MAX_DEVICES) return fail(FG_ERR_UNSUPPORTED, "%s: device %d beyond %d", fn, dev, MAX_DEVICES);
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return fail(FG_ERR_HIP, "%s: hipGetSymbolAddress of the static scratch failed: %s", fn,
                    hipGetErrorString(e));
      }
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return FG_OK;
}

}  // namespace fg

using namespace fg;

extern "C" size_t moe_noalloc_scratch_bytes(void) { return MOE_SCRATCH_BYTES; }

extern "C" fg_status moe_grouped_ffn_noalloc(const moe_desc* d, const void* tokens, const float* router_logits,
                                             const void* w_gateup, const void* w_down, const float* s_gateup,
                                             const float* s_down, void* out, int32_t* topk_idx, float* topk_w,
                                             int32_t* perm, int32_t* expert_offsets, void* stream) {
  clear_error();
  const char* fn = "moe_grouped_ffn_noalloc";
  const fg_status st = validate_desc(d, fn);
  if (st != FG_OK) return st;
  const size_t need = moe_workspace_bytes(d);
  if (need > MOE_SCRATCH_BYTES)
    return fail(FG_ERR_UNSUPPORTED,
                "%s: this problem needs %zu bytes of scratch; the static scratch holds %zu (use "
                "moe_grouped_ffn with a workspace)",
                fn, need, MOE_SCRATCH_BYTES);
  void* ws = nullptr;
  const fg_status sst = scratch_on_device(fn, &ws);
  if (sst != FG_OK) return sst;
  return moe_run(fn, d, tokens, router_logits, w_gateup, w_down, s_gateup, s_down, out, topk_idx, topk_w, perm,
                 expert_offsets, ws, MOE_SCRATCH_BYTES, stream);
}
