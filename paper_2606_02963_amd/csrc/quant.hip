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

__global__ __launch_bounds__(256) void quantize_rows_kernel(const uint16_t* x, int64_t rows, int64_t cols,
                                                            uint8_t* q, float* s) {
  quantize_row_wave(x, rows, cols, q, s, (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
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
  Launches lc;
  lc.add(launch(quantize_rows_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                static_cast<const uint16_t*>(x), rows, cols, q, s));
  return check_launch("fg_quantize_rows_e4m3", lc);
}
