// moe.hip — MoE expert FFN step (placeholder entry points; kernels follow).
#include <hip/hip_runtime.h>

#include "fg_host.hpp"
#include "fgemm.h"

using namespace fg;

extern "C" size_t moe_workspace_bytes(const moe_desc* d) {
  (void)d;
  return 0;
}

extern "C" fg_status moe_grouped_ffn(const moe_desc* d, const void* tokens, const float* router_logits,
                                     const void* w_gateup, const void* w_down, const float* s_gateup,
                                     const float* s_down, void* out, int32_t* topk_idx, float* topk_w,
                                     int32_t* perm, int32_t* expert_offsets, void* workspace, size_t ws_bytes,
                                     void* stream) {
  clear_error();
  (void)d; (void)tokens; (void)router_logits; (void)w_gateup; (void)w_down; (void)s_gateup; (void)s_down;
  (void)out; (void)topk_idx; (void)topk_w; (void)perm; (void)expert_offsets; (void)workspace;
  (void)ws_bytes; (void)stream;
  return fail(FG_ERR_UNSUPPORTED, "moe_grouped_ffn: not built yet");
}
