// fg_quant.hpp — device helpers for OCP e4m3fn quantisation.
#pragma once

#include <hip/hip_runtime.h>

#include "fg_tile.hpp"

namespace fg {

constexpr float E4M3_MAX = 448.0f;

// Per-row scale s = amax/448 (correctly rounded fp32 division); an all-zero
// row gets s = 1 so that v/s stays 0.
__device__ __forceinline__ float e4m3_row_scale(float amax) {
  return amax > 0.0f ? amax / E4M3_MAX : 1.0f;
}

// Saturate to ±448, then round to nearest even into e4m3fn
// (v_cvt_pk_fp8_f32 uses the OCP e4m3 encoding on gfx950); four values are
// packed little-endian into one 32-bit word.
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d) {
  a = fminf(fmaxf(a, -E4M3_MAX), E4M3_MAX);
  b = fminf(fmaxf(b, -E4M3_MAX), E4M3_MAX);
  c = fminf(fmaxf(c, -E4M3_MAX), E4M3_MAX);
  d = fminf(fmaxf(d, -E4M3_MAX), E4M3_MAX);
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

}  // namespace fg
