// fg_moe.hpp — the MoE step's host-side body, shared by moe_grouped_ffn
// (caller's workspace) and moe_grouped_ffn_noalloc (the library's static
// scratch).
#pragma once

#include "fgemm.h"

namespace fg {

// Checks the descriptor; FG_OK or the status fg_last_error describes.
fg_status validate_desc(const moe_desc* d, const char* fn);

// Validates every argument (workspace of at least moe_workspace_bytes(d)
// included) and enqueues the step on `stream`; `fn` names the entry point in
// error messages.
fg_status moe_run(const char* fn, const moe_desc* d, const void* tokens, const float* router_logits,
                  const void* w_gateup, const void* w_down, const float* s_gateup, const float* s_down, void* out,
                  int32_t* topk_idx, float* topk_w, int32_t* perm, int32_t* expert_offsets, void* workspace,
                  size_t ws_bytes, void* stream);

}  // namespace fg
