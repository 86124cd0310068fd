// quant.hip — per-row e4m3 (OCP e4m3fn) quantisation of bf16 activations.
//
// The W8A8 variant of the MoE FFN quantises activations on the fly with one
// fp32 scale per row: s = amax/448 (1 for an all-zero row), code =
// RNE_sat(v/s). Both decisions are taken in fp32: the division is the
// correctly rounded fp32 quotient and the conversion rounds to nearest even
// after saturating to ±448, the largest finite e4m3fn value.
#include <hip/hip_runtime.h>

#include "fg_host.hpp"
#include "fg_quant.hpp"
#include "fgemm.h"

namespace fg {

// One wave per row; each lane handles 8-value chunks l, l + 64, ... Rows of
// up to 64·REG chunks are loaded once, with every load in flight together,
// and quantised from the registers; longer rows take a second pass that
// reads the row again.
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

__global__ __launch_bounds__(256) void quantize_rows_kernel(const uint16_t* x, int64_t rows, int64_t cols,
                                                            uint8_t* q, float* s) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
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

using namespace fg;

extern "C" fg_status fg_quantize_rows_e4m3(const void* x, int64_t rows, int64_t cols, uint8_t* q, float* s,
                                           void* stream) {
  clear_error();
  if (rows < 0 || cols <= 0 || rows > 0x7fffffffLL * 4 || cols > 0x7fffffffLL)
    return fail(FG_ERR_INVALID_ARG, "fg_quantize_rows_e4m3: bad shape %lld x %lld", (long long)rows,
                (long long)cols);
  if (cols % 8 != 0) return fail(FG_ERR_ALIGNMENT, "fg_quantize_rows_e4m3: cols must be a multiple of 8");
  if (rows == 0) return FG_OK;
  if (x == nullptr || q == nullptr || s == nullptr)
    return fail(FG_ERR_INVALID_ARG, "fg_quantize_rows_e4m3: NULL pointer");
  if (!aligned16(x) || (reinterpret_cast<uintptr_t>(q) & 7u) != 0 || (reinterpret_cast<uintptr_t>(s) & 3u) != 0)
    return fail(FG_ERR_ALIGNMENT, "fg_quantize_rows_e4m3: x must be 16-byte and q 8-byte aligned");
  const unsigned grid = (unsigned)((rows + 3) / 4);
  hipLaunchKernelGGL(quantize_rows_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint16_t*>(x), rows, cols, q, s);
  return check_launch("fg_quantize_rows_e4m3");
}
