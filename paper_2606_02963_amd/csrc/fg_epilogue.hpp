// fg_epilogue.hpp — the in-register tail applied to fp32 accumulator tiles.
//
// The post-GEMM sequence runs on the accumulators before the single store
// (paper §IV-B, layer-wise fusion and fp32 post-processing). Elementwise ops
// are applied one op at a time over the whole tile, so the branch on the op
// kind is uniform across the workgroup. Row reductions follow the
// single-pass pattern of §IV-B: GroupNorm groups never straddle a tile, so
// mean and variance come from the registers plus one exchange between the
// two waves that share a row; LogSumExp spans N tiles, so each tile emits its
// (max, Σexp) pair and a second, tiny pass combines them with the rescaling
// identity of online softmax (§I). Table III also chains elementwise ops
// after the reduction (LSE → Mish, GroupNorm → Swish → Mul → Swish); those
// run on the normalised registers, or on the combined row value.
#pragma once

#include <math.h>

#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

struct EpiArgs {
  int32_t n_ops;
  int32_t kind[FG_MAX_OPS];
  float a[FG_MAX_OPS];
  float b[FG_MAX_OPS];
};

// GELU, tanh form: ½u(1 + tanh(z)) with z = √(2/π)(u + 0.044715u³). Since
// ½(1 + tanh z) = σ(2z), this is u·σ(2z): one exponential and one
// reciprocal instead of a tanh.
__device__ __forceinline__ float gelu_tanh(float u) {
  const float k0 = 2.0f * 0.7978845608028654f;  // 2·√(2/π)
  const float k1 = 0.044715f;
  return u * fast_sigmoid(k0 * (u + k1 * u * u * u));
}

// SiLU u·σ(u); for u → −∞ it tends to −0.
__device__ __forceinline__ float silu(float u) { return u * fast_sigmoid(u); }

// Mish u·tanh(ln(1 + e^u)). With t = e^u, tanh(ln(1 + t)) = n/(n + 2) where
// n = (1 + t)² − 1 = t(t + 2): one exponential and one reciprocal. Above
// u = 20 the ratio is 1 in fp32, and clamping the exponent there keeps n
// finite (n overflows near u = 44).
__device__ __forceinline__ float mish(float u) {
  const float t = fast_exp(fminf(u, 20.0f));
  const float n = t * (t + 2.0f);
  return u * (n * fast_rcp(n + 2.0f));
}

__device__ __forceinline__ float leaky_relu(float u, float slope) { return u >= 0.0f ? u : slope * u; }

// One op on one value: the per-row values after a row LogSumExp.
__device__ __forceinline__ float apply_op_scalar(int kind, float a, float b, float u) {
  switch (kind) {
    case FG_OP_SCALE: return u * a;
    case FG_OP_ADD: return u + a;
    case FG_OP_RELU: return fmaxf(u, 0.0f);
    case FG_OP_GELU_TANH: return gelu_tanh(u);
    case FG_OP_SILU: return silu(u);
    case FG_OP_CLAMP: return fminf(fmaxf(u, a), b);
    case FG_OP_MISH: return mish(u);
    case FG_OP_LEAKY_RELU: return leaky_relu(u, a);
    default: return u;
  }
}

// The chain runs over one block of FN·4 accumulators at a time (one fm),
// all ops on that block before the next, so only that block's temporaries
// (the transcendental intermediates) are live beside the accumulators.
template <class TL>
__device__ __forceinline__ void apply_ops(const EpiArgs& ep, f32x4 (&acc)[TL::FM][TL::FN]) {
  if (ep.n_ops == 0) return;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm) {
    float v[TL::FN * 4];
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
      for (int i = 0; i < 4; ++i) v[fn * 4 + i] = acc[fm][fn][i];
    for (int o = 0; o < ep.n_ops; ++o) {
      const int kind = ep.kind[o];
      const float a = ep.a[o], b = ep.b[o];
#define FG_EACH(EXPR)                                           \
  _Pragma("unroll") for (int e = 0; e < TL::FN * 4; ++e) {      \
    const float u = v[e];                                       \
    v[e] = (EXPR);                                              \
  }
      switch (kind) {
        case FG_OP_SCALE: FG_EACH(u * a) break;
        case FG_OP_ADD: FG_EACH(u + a) break;
        case FG_OP_RELU: FG_EACH(fmaxf(u, 0.0f)) break;
        case FG_OP_GELU_TANH: FG_EACH(gelu_tanh(u)) break;
        case FG_OP_SILU: FG_EACH(silu(u)) break;
        case FG_OP_CLAMP: FG_EACH(fminf(fmaxf(u, a), b)) break;
        case FG_OP_MISH: FG_EACH(mish(u)) break;
        case FG_OP_LEAKY_RELU: FG_EACH(leaky_relu(u, a)) break;
        default: break;
      }
#undef FG_EACH
    }
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[fm][fn][i] = v[fn * 4 + i];
  }
}

// Add bias[n0 + col] (columns past N read nothing and add 0).
template <class TL>
__device__ __forceinline__ void add_bias(const float* bias, int n0, int N, f32x4 (&acc)[TL::FM][TL::FN]) {
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int n = n0 + acc_col<TL>(fn);
    const float bv = n < N ? bias[n] : 0.0f;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[fm][fn][i] += bv;
  }
}

// Per-tile row LogSumExp partials: for every tile row r, over the tile's
// valid columns, m = max t and s = Σ exp(t − m). `red` needs 2·WN·BM floats
// of LDS. Rows ≥ M are skipped. ws is [M, tiles_n] (m, s) pairs.
template <class TL>
__device__ __forceinline__ void lse_partials(f32x4 (&acc)[TL::FM][TL::FN], float* red, int m0, int n0,
                                             int M, int N, int tn, int tiles_n, float2* ws) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int wn = wave % TL::WN;
  float* rmax = red;
  float* rsum = red + TL::WN * TL::BM;
  bool colok[TL::FN];
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) colok[fn] = n0 + acc_col<TL>(fn) < N;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = -INFINITY;
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        if (colok[fn]) mx = fmaxf(mx, acc[fm][fn][i]);
      mx = row16_max(mx);
      if ((l & 15) == 0) rmax[wn * TL::BM + acc_row<TL>(fm, i)] = mx;
    }
  __syncthreads();
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = acc_row<TL>(fm, i);
      float mx = rmax[r];
#pragma unroll
      for (int w = 1; w < TL::WN; ++w) mx = fmaxf(mx, rmax[w * TL::BM + r]);
      float s = 0.0f;
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        if (colok[fn]) s += fast_exp(acc[fm][fn][i] - mx);
      s = row16_sum(s);
      if ((l & 15) == 0) rsum[wn * TL::BM + r] = s;
    }
  __syncthreads();
  // one thread per tile row writes the pair
  for (int r = threadIdx.x; r < TL::BM; r += TL::THREADS) {
    if (m0 + r >= M) continue;
    float mx = rmax[r], s = 0.0f;
#pragma unroll
    for (int w = 1; w < TL::WN; ++w) mx = fmaxf(mx, rmax[w * TL::BM + r]);
#pragma unroll
    for (int w = 0; w < TL::WN; ++w) s += rsum[w * TL::BM + r];
    ws[(int64_t)(m0 + r) * tiles_n + tn] = make_float2(mx, s);
  }
}

// Sum over the 16 lanes of a DPP row that every lane receives bit for bit:
// quad_perm [1,0,3,2] and [2,3,0,1], then row_half_mirror and row_mirror
// pair each lane with a partner holding the same partial sums in the same
// association, so the final value does not depend on the lane.
__device__ __forceinline__ float row16_sum_uniform(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  return v;
}

// GroupNorm over groups of FPG whole 16-column fragments of one wave
// (gw = 16·FPG ≤ TN): each group's mean, then its biased variance about the
// mean, from the wave's registers with one 16-lane reduction per row and
// group; then the normalisation and the per-channel affine map.
template <class TL, int FPG>
__device__ __forceinline__ void groupnorm_inwave(f32x4 (&acc)[TL::FM][TL::FN], int n0, int N, float eps,
                                                 const float* gamma, const float* beta) {
  static_assert(TL::FN % FPG == 0, "a group must be whole fragments of one wave");
  constexpr float inv_gw = 1.0f / (16.0f * FPG);
  float gm[TL::FN], bt[TL::FN];
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int n = n0 + acc_col<TL>(fn);
    gm[fn] = n < N ? gamma[n] : 0.0f;
    bt[fn] = n < N ? beta[n] : 0.0f;
  }
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < TL::FN / FPG; ++q) {
        float sm = 0.0f;
#pragma unroll
        for (int f = 0; f < FPG; ++f) sm += acc[fm][q * FPG + f][i];
        const float mu = row16_sum_uniform(sm) * inv_gw;
        float sq = 0.0f;
#pragma unroll
        for (int f = 0; f < FPG; ++f) {
          const float d = acc[fm][q * FPG + f][i] - mu;
          sq += d * d;
        }
        const float rstd = fast_rsqrt(row16_sum_uniform(sq) * inv_gw + eps);
#pragma unroll
        for (int f = 0; f < FPG; ++f) {
          const int fn = q * FPG + f;
          acc[fm][fn][i] = (acc[fm][fn][i] - mu) * rstd * gm[fn] + bt[fn];
        }
      }
}

// Whether a tile can normalise groups of gw channels in registers: gw a
// multiple of 16 that either divides the wave tile width (a group is whole
// fragments of one wave) or is a multiple of it that divides the tile width
// (a group is whole wave columns).
template <class TL>
constexpr bool groupnorm_fits_tile(int gw) {
  return gw % 16 == 0 && (gw <= TL::TN ? TL::TN % gw == 0 : (gw % TL::TN == 0 && TL::BN % gw == 0));
}

// GroupNorm inside the tile, for groups that groupnorm_fits_tile accepts.
// Groups of at most one wave's width are handled by groupnorm_inwave; wider
// groups span whole wave columns, and their statistics are the sum over the
// waves whose columns they cover (exchanged through `red`, WN·BM floats of
// LDS). Both take the mean first and then the biased variance about it.
template <class TL>
__device__ __forceinline__ void groupnorm_tile(f32x4 (&acc)[TL::FM][TL::FN], float* red, int n0, int N,
                                               int gw, float eps, const float* gamma, const float* beta) {
  static_assert(TL::FN == 4, "the in-wave group sizes below assume 64-column wave tiles");
  if (gw <= TL::TN) {
    // 16, 32 or 64 channels (the host admits no other width here)
    if (gw == 16)
      groupnorm_inwave<TL, 1>(acc, n0, N, eps, gamma, beta);
    else if (gw == 32)
      groupnorm_inwave<TL, 2>(acc, n0, N, eps, gamma, beta);
    else
      groupnorm_inwave<TL, 4>(acc, n0, N, eps, gamma, beta);
    return;
  }
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int wn = wave % TL::WN;
  const int my_group = (wn * TL::TN) / gw;
  const float inv_gw = 1.0f / (float)gw;
  float mean[TL::FM][4];
  // pass 1: mean
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = 0.0f;
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) s += acc[fm][fn][i];
      s = row16_sum(s);
      if ((l & 15) == 0) red[wn * TL::BM + acc_row<TL>(fm, i)] = s;
    }
  __syncthreads();
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = acc_row<TL>(fm, i);
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < TL::WN; ++w)
        if ((w * TL::TN) / gw == my_group) s += red[w * TL::BM + r];
      mean[fm][i] = s * inv_gw;
    }
  __syncthreads();
  // pass 2: biased variance about the mean
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = 0.0f;
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) {
        const float d = acc[fm][fn][i] - mean[fm][i];
        s += d * d;
      }
      s = row16_sum(s);
      if ((l & 15) == 0) red[wn * TL::BM + acc_row<TL>(fm, i)] = s;
    }
  __syncthreads();
  float gm[TL::FN], bt[TL::FN];
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int n = n0 + acc_col<TL>(fn);
    gm[fn] = n < N ? gamma[n] : 0.0f;
    bt[fn] = n < N ? beta[n] : 0.0f;
  }
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = acc_row<TL>(fm, i);
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < TL::WN; ++w)
        if ((w * TL::TN) / gw == my_group) s += red[w * TL::BM + r];
      const float rstd = fast_rsqrt(s * inv_gw + eps);
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        acc[fm][fn][i] = (acc[fm][fn][i] - mean[fm][i]) * rstd * gm[fn] + bt[fn];
    }
}

}  // namespace fg
