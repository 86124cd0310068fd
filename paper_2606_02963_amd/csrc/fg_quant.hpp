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

// Row quantisation, one wave per row: each lane handles 8-value chunks
// l, l + 64, ... Rows of up to 64·QUANT_REG chunks are loaded once, with every
// load in flight together, and quantised from the registers; longer rows take
// a second pass that reads the row again.
constexpr int QUANT_REG = 8;

__device__ __forceinline__ float chunk_amax(const i32x4& v, float amax) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    amax = fmaxf(amax, fabsf(bf16_bits_to_f32((uint16_t)(v[j] & 0xffff))));
    amax = fmaxf(amax, fabsf(bf16_bits_to_f32((uint16_t)((uint32_t)v[j] >> 16))));
  }
  return amax;
}

__device__ __forceinline__ uint2 chunk_quant(const i32x4& v, float sc) {
  float f[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f[2 * j] = bf16_bits_to_f32((uint16_t)(v[j] & 0xffff));
    f[2 * j + 1] = bf16_bits_to_f32((uint16_t)((uint32_t)v[j] >> 16));
  }
  uint2 packed;
  packed.x = e4m3_pack4(f[0] / sc, f[1] / sc, f[2] / sc, f[3] / sc);
  packed.y = e4m3_pack4(f[4] / sc, f[5] / sc, f[6] / sc, f[7] / sc);
  return packed;
}

// Quantise row `row` of x [rows, cols] (bf16) into q (e4m3 codes, same
// layout) and s[row]; rows ≥ `rows` do nothing. Called by a whole wave.
__device__ __forceinline__ void quantize_row_wave(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q,
                                                  float* s, int64_t row) {
  const int l = threadIdx.x & 63;
  if (row >= rows) return;
  const uint16_t* xr = x + row * cols;
  uint8_t* qr = q + row * cols;
  const int64_t nch = cols / 8;
  float amax = 0.0f;
  if (nch <= 64 * QUANT_REG) {
    i32x4 v[QUANT_REG];
#pragma unroll
    for (int u = 0; u < QUANT_REG; ++u) {
      const int64_t c = l + 64 * u;
      v[u] = c < nch ? *reinterpret_cast<const i32x4*>(xr + c * 8) : i32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < QUANT_REG; ++u) amax = chunk_amax(v[u], amax);
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 64));
    const float sc = e4m3_row_scale(amax);
    if (l == 0) s[row] = sc;
#pragma unroll
    for (int u = 0; u < QUANT_REG; ++u) {
      const int64_t c = l + 64 * u;
      if (c < nch) *reinterpret_cast<uint2*>(qr + c * 8) = chunk_quant(v[u], sc);
    }
    return;
  }
  for (int64_t c = l; c < nch; c += 64) amax = chunk_amax(*reinterpret_cast<const i32x4*>(xr + c * 8), amax);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) amax = fmaxf(amax, __shfl_xor(amax, m, 64));
  const float sc = e4m3_row_scale(amax);
  if (l == 0) s[row] = sc;
  for (int64_t c = l; c < nch; c += 64)
    *reinterpret_cast<uint2*>(qr + c * 8) = chunk_quant(*reinterpret_cast<const i32x4*>(xr + c * 8), sc);
}

}  // namespace fg
