// norm.hip — fused residual add + RMSNorm of the gpt-oss-20b decode path
// (paper §IV-A, "Fused Add + RMSNorm" in Table I).
//
//   s = x + residual (fp32; exact for bf16 inputs)
//   residual ← bf16(s)                      (RNE, in place)
//   out      = bf16(s · rsqrt(mean(s²) + eps) · weight)
//
// One workgroup of 256 threads per row; thread i holds 8-value chunks i,
// i + 256, ... of the row in registers, so every load of the row (x, residual
// and weight chunks) is in flight together and the row is read once: one
// memory round trip, a few values of arithmetic per lane, one reduction (DPP
// inside each 16-lane row, the four row sums of a wave as scalars, the four
// wave sums through LDS), then the stores. Rows of up to 256·NORM_REG chunks
// (4096 values).
#include <hip/hip_runtime.h>
#include <math.h>

#include "fg_host.hpp"
#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

constexpr int NORM_REG = 2;
constexpr int NORM_THREADS = 256;
constexpr int64_t NORM_MAX_H = NORM_THREADS * NORM_REG * 8;

__device__ __forceinline__ void unpack8(const i32x4& v, float (&f)[8]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f[2 * q] = bf16_bits_to_f32((uint16_t)(v[q] & 0xffff));
    f[2 * q + 1] = bf16_bits_to_f32((uint16_t)((uint32_t)v[q] >> 16));
  }
}

__device__ __forceinline__ i32x4 pack8(const float (&f)[8]) {
  i32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = (int)((uint32_t)f32_to_bf16_bits(f[2 * q]) | ((uint32_t)f32_to_bf16_bits(f[2 * q + 1]) << 16));
  return o;
}

__device__ __forceinline__ float wave_sum(float v) {
  v = row16_sum(v);
  const int vi = __builtin_bit_cast(int, v);
  return (__builtin_bit_cast(float, __builtin_amdgcn_readlane(vi, 0)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(vi, 16))) +
         (__builtin_bit_cast(float, __builtin_amdgcn_readlane(vi, 32)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(vi, 48)));
}

__global__ __launch_bounds__(NORM_THREADS) void add_rmsnorm_kernel(const uint16_t* x, uint16_t* res,
                                                                   const uint16_t* w, uint16_t* out, int H,
                                                                   float eps) {
  __shared__ float part[NORM_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * H;
  const int nch = H / 8;
  i32x4 xv[NORM_REG], rv[NORM_REG], wv[NORM_REG];
#pragma unroll
  for (int u = 0; u < NORM_REG; ++u) {
    const int c = threadIdx.x + NORM_THREADS * u;
    const bool in = c < nch;
    xv[u] = in ? *reinterpret_cast<const i32x4*>(x + base + c * 8) : i32x4{0, 0, 0, 0};
    rv[u] = in ? *reinterpret_cast<const i32x4*>(res + base + c * 8) : i32x4{0, 0, 0, 0};
    wv[u] = in ? *reinterpret_cast<const i32x4*>(w + c * 8) : i32x4{0, 0, 0, 0};
  }
  float s[NORM_REG][8];
  float ss = 0.0f;
#pragma unroll
  for (int u = 0; u < NORM_REG; ++u) {
    float a[8], b[8];
    unpack8(xv[u], a);
    unpack8(rv[u], b);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s[u][i] = a[i] + b[i];
      ss = fmaf(s[u][i], s[u][i], ss);
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = (part[0] + part[1]) + (part[2] + part[3]);
  const float inv = 1.0f / sqrtf(ss / (float)H + eps);
#pragma unroll
  for (int u = 0; u < NORM_REG; ++u) {
    const int c = threadIdx.x + NORM_THREADS * u;
    if (c < nch) {
      float g[8], o[8];
      unpack8(wv[u], g);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = s[u][i] * inv * g[i];
      *reinterpret_cast<i32x4*>(res + base + c * 8) = pack8(s[u]);
      *reinterpret_cast<i32x4*>(out + base + c * 8) = pack8(o);
    }
  }
}

}  // namespace fg

using namespace fg;

extern "C" fg_status add_rmsnorm(const void* x, void* residual, const void* weight, void* out, int64_t T, int64_t H,
                                 float eps, void* stream) {
  clear_error();
  const char* fn = "add_rmsnorm";
  if (T < 0 || T > 0x7fffffffLL || H <= 0)
    return fail(FG_ERR_INVALID_ARG, "%s: bad T=%lld or H=%lld", fn, (long long)T, (long long)H);
  if (!(eps >= 0.0f) || !isfinite(eps)) return fail(FG_ERR_INVALID_ARG, "%s: eps must be finite and >= 0", fn);
  if (H % 8 != 0) return fail(FG_ERR_ALIGNMENT, "%s: H must be a multiple of 8", fn);
  if (H > NORM_MAX_H) return fail(FG_ERR_UNSUPPORTED, "%s: H=%lld above %lld", fn, (long long)H, (long long)NORM_MAX_H);
  if (T == 0) return FG_OK;
  if (x == nullptr || residual == nullptr || weight == nullptr || out == nullptr)
    return fail(FG_ERR_INVALID_ARG, "%s: NULL pointer", fn);
  if (!aligned16(x) || !aligned16(residual) || !aligned16(weight) || !aligned16(out))
    return fail(FG_ERR_ALIGNMENT, "%s: pointers must be 16-byte aligned", fn);
  Launches lc;
  lc.add(launch(add_rmsnorm_kernel, dim3((unsigned)T), dim3(NORM_THREADS), 0, static_cast<hipStream_t>(stream),
                static_cast<const uint16_t*>(x), static_cast<uint16_t*>(residual),
                static_cast<const uint16_t*>(weight), static_cast<uint16_t*>(out), (int)H, eps));
  return check_launch(fn, lc);
}
