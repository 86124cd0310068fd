// fgemm.hip — the fused dense GEMM + tail: y = tail(x·Wᵀ + b).
//
// One kernel launch computes the GEMM on the matrix cores and applies the
// whole tail on the fp32 accumulators before its single store (paper §IV-B:
// layer-wise fusion, fp32 accumulation and post-processing). The one
// exception is a LogSumExp over a row that spans several N tiles: each tile
// writes its (max, Σexp) pair and a second launch of one wave per row
// combines them (the rescaling identity of online softmax, §I).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <new>

#include "fg_epilogue.hpp"
#include "fg_host.hpp"
#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

enum : int { OUT_F32 = 0, OUT_BF16 = 1 };

template <class TL>
struct DenseLds {
  static constexpr int OUT_STAGE = TL::BM * (TL::BN * 2 + 16);
  static constexpr int MAIN = TL::LOOP_LDS > OUT_STAGE ? TL::LOOP_LDS : OUT_STAGE;
  static constexpr int RED = 2 * TL::WN * TL::BM * 4;
  static constexpr int BYTES = MAIN + RED;
};

struct DenseArgs {
  const char* A;
  const char* W;
  const float* bias;
  const float* gamma;
  const float* beta;
  void* out;
  float2* ws;
  int M, N;
  int64_t K;
  int tiles_n;
  int gn_width;
  float gn_eps;
};

template <class TL, int RED, int OUT>
__global__ __launch_bounds__(TL::THREADS) void fgemm_kernel(DenseArgs a, EpiArgs ep) {
  __shared__ __attribute__((aligned(16))) char lds[DenseLds<TL>::BYTES];
  const int tm = blockIdx.x / a.tiles_n, tn = blockIdx.x % a.tiles_n;
  const int m0 = tm * TL::BM, n0 = tn * TL::BN;
  const int64_t rowbytes = a.K * TL::ESIZE;
  const int r0 = threadIdx.x >> 3;

  RowSet<TL::A_LD> ra;
  RowSet<TL::B_LD> rb;
#pragma unroll
  for (int p = 0; p < TL::A_LD; ++p) {
    const int m = m0 + r0 + TL::RSTRIDE * p;
    ra.ptr[p] = a.A + (int64_t)(m < a.M ? m : a.M - 1) * rowbytes;
  }
#pragma unroll
  for (int p = 0; p < TL::B_LD; ++p) {
    const int n = n0 + r0 + TL::RSTRIDE * p;
    rb.ptr[p] = a.W + (int64_t)(n < a.N ? n : a.N - 1) * rowbytes;
  }

  f32x4 acc[TL::FM][TL::FN];
  gemm_mainloop<TL>(ra, rb, rowbytes, lds, acc);

  if (a.bias != nullptr) add_bias<TL>(a.bias, n0, a.N, acc);
  apply_ops<TL>(ep, acc);

  float* red = reinterpret_cast<float*>(lds + DenseLds<TL>::MAIN);
  if constexpr (RED == FG_RED_LOGSUMEXP_ROW) {
    lse_partials<TL>(acc, red, m0, n0, a.M, a.N, tn, a.tiles_n, a.ws);
    return;
  }
  if constexpr (RED == FG_RED_GROUPNORM)
    groupnorm_tile<TL>(acc, red, n0, a.N, a.gn_width, a.gn_eps, a.gamma, a.beta);

  if constexpr (OUT == OUT_BF16) {
    char* out = reinterpret_cast<char*>(a.out);
    const int ncols = a.N - n0 < TL::BN ? a.N - n0 : TL::BN;
    store_tile_bf16<TL, TL::BN>(
        lds,
        [&](int fm, int fn, int i, float& v, int& c) {
          v = acc[fm][fn][i];
          c = acc_col<TL>(fn);
          return true;
        },
        [&](int r) -> char* {
          const int m = m0 + r;
          return m < a.M ? out + ((int64_t)m * a.N + n0) * 2 : nullptr;
        },
        ncols);
  } else {
    float* out = reinterpret_cast<float*>(a.out);
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) {
        const int n = n0 + acc_col<TL>(fn);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + acc_row<TL>(fm, i);
          if (m < a.M && n < a.N) out[(int64_t)m * a.N + n] = acc[fm][fn][i];
        }
      }
  }
}

// out[m] = max_j m_j + log Σ_j s_j·exp(m_j − max_j m_j); one wave per row.
__global__ __launch_bounds__(256) void lse_combine_kernel(const float2* ws, float* out, int M, int tiles_n) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (row >= M) return;
  const float2* p = ws + (int64_t)row * tiles_n;
  float mx = -INFINITY;
  for (int j = l; j < tiles_n; j += 64) mx = fmaxf(mx, p[j].x);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
  float s = 0.0f;
  for (int j = l; j < tiles_n; j += 64) s += p[j].y * expf(p[j].x - mx);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) s += __shfl_xor(s, m, 64);
  if (l == 0) out[row] = mx + logf(s);
}

// ---------------------------------------------------------------------------
// kernel table

typedef Tile<In::F32, 64, 128> TileF32;
typedef Tile<In::BF16, 256, 128, 4, 2> TileBig;
typedef Tile<In::BF16, 128, 128> TileMid;

enum Cfg : int { CFG_F32 = 0, CFG_BF16_256x128 = 1, CFG_BF16_128x128 = 2 };

typedef void (*KernelFn)(DenseArgs, EpiArgs);

struct KernelChoice {
  KernelFn fn;
  int threads;
};

template <class TL>
static KernelChoice pick_kernel(int red, int out) {
  KernelFn fn = nullptr;
  switch (red) {
    case FG_RED_NONE:
      fn = out == OUT_BF16 ? fgemm_kernel<TL, FG_RED_NONE, OUT_BF16> : fgemm_kernel<TL, FG_RED_NONE, OUT_F32>;
      break;
    case FG_RED_LOGSUMEXP_ROW:
      fn = fgemm_kernel<TL, FG_RED_LOGSUMEXP_ROW, OUT_F32>;
      break;
    case FG_RED_GROUPNORM:
      fn = out == OUT_BF16 ? fgemm_kernel<TL, FG_RED_GROUPNORM, OUT_BF16>
                           : fgemm_kernel<TL, FG_RED_GROUPNORM, OUT_F32>;
      break;
  }
  return KernelChoice{fn, TL::THREADS};
}

}  // namespace fg

using namespace fg;

struct fg_plan {
  int64_t M, N, K;
  int32_t in_dt, out_dt;
  fg_epilogue epi;
  int cfg;
  int BM, BN;
  int64_t tiles_m, tiles_n;
  size_t ws_bytes;
};

extern "C" fg_status fgemm_plan(fg_plan** plan, int64_t M, int64_t N, int64_t K, int32_t in_dtype,
                                int32_t out_dtype, const fg_epilogue* epi) {
  clear_error();
  if (plan == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan: plan is NULL");
  *plan = nullptr;
  if (epi == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan: epi is NULL");
  const int64_t LIM = 0x7fffffffLL;
  if (M < 0 || N <= 0 || K < 0 || M > LIM || N > LIM || K > LIM)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: bad shape M=%lld N=%lld K=%lld", (long long)M,
                (long long)N, (long long)K);
  if (in_dtype != FG_F32 && in_dtype != FG_BF16)
    return fail(in_dtype == FG_E4M3 ? FG_ERR_UNSUPPORTED : FG_ERR_INVALID_ARG,
                "fgemm_plan: input dtype %d not supported (f32 or bf16)", in_dtype);
  if (out_dtype != FG_F32 && out_dtype != FG_BF16)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: output dtype %d not supported (f32 or bf16)", out_dtype);
  if (epi->n_ops < 0 || epi->n_ops > FG_MAX_OPS)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: n_ops=%d outside 0..%d", epi->n_ops, FG_MAX_OPS);
  for (int i = 0; i < epi->n_ops; ++i) {
    const fg_op& op = epi->ops[i];
    if (op.kind < FG_OP_SCALE || op.kind > FG_OP_CLAMP)
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: op %d has unknown kind %d", i, op.kind);
    if (op.kind == FG_OP_CLAMP && !(op.a <= op.b))
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: clamp op %d needs lo <= hi", i);
    if (!isfinite(op.a) || !isfinite(op.b))
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: op %d has a non-finite parameter", i);
  }
  if (epi->has_bias != 0 && epi->has_bias != 1)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: has_bias must be 0 or 1");
  const int red = epi->reduction;
  if (red != FG_RED_NONE && red != FG_RED_LOGSUMEXP_ROW && red != FG_RED_GROUPNORM)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: unknown reduction %d", red);
  if (red == FG_RED_LOGSUMEXP_ROW && out_dtype != FG_F32)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: LogSumExp output must be f32");
  const int epc = in_dtype == FG_F32 ? 4 : 8;
  if (K % epc != 0)
    return fail(FG_ERR_ALIGNMENT, "fgemm_plan: K=%lld must be a multiple of %d", (long long)K, epc);
  if (red != FG_RED_LOGSUMEXP_ROW) {
    const int opc = out_dtype == FG_F32 ? 4 : 8;
    if (N % opc != 0)
      return fail(FG_ERR_ALIGNMENT, "fgemm_plan: N=%lld must be a multiple of %d", (long long)N, opc);
  }
  int gw = 0;
  if (red == FG_RED_GROUPNORM) {
    if (epi->gn_groups <= 0 || N % epi->gn_groups != 0)
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: N=%lld not divisible into %d groups", (long long)N,
                  epi->gn_groups);
    if (!(epi->gn_eps >= 0.0f) || !isfinite(epi->gn_eps))
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: gn_eps must be finite and >= 0");
    gw = (int)(N / epi->gn_groups);
    if (gw != 64 && gw != 128)
      return fail(FG_ERR_UNSUPPORTED, "fgemm_plan: GroupNorm group width %d (supported: 64, 128)", gw);
  }

  fg_plan* p = new (std::nothrow) fg_plan();
  if (p == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan: out of host memory");
  p->M = M;
  p->N = N;
  p->K = K;
  p->in_dt = in_dtype;
  p->out_dt = out_dtype;
  p->epi = *epi;
  if (in_dtype == FG_F32) {
    p->cfg = CFG_F32;
    p->BM = TileF32::BM;
    p->BN = TileF32::BN;
  } else {
    // The 256×128 tile halves the operand traffic per FLOP against 128×128;
    // use it whenever it still yields at least one tile per compute unit.
    const int64_t big_tiles = ((M + 255) / 256) * ((N + 127) / 128);
    if (big_tiles >= 256) {
      p->cfg = CFG_BF16_256x128;
      p->BM = 256;
      p->BN = 128;
    } else {
      p->cfg = CFG_BF16_128x128;
      p->BM = 128;
      p->BN = 128;
    }
  }
  p->tiles_m = (M + p->BM - 1) / p->BM;
  p->tiles_n = (N + p->BN - 1) / p->BN;
  if (p->tiles_m * p->tiles_n > LIM) {
    delete p;
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: too many tiles");
  }
  p->ws_bytes = red == FG_RED_LOGSUMEXP_ROW ? (size_t)M * (size_t)p->tiles_n * sizeof(float2) : 0;
  *plan = p;
  return FG_OK;
}

extern "C" size_t fgemm_workspace_bytes(const fg_plan* plan) { return plan ? plan->ws_bytes : 0; }

extern "C" void fgemm_destroy(fg_plan* plan) { delete plan; }

extern "C" fg_status fgemm_plan_info(const fg_plan* plan, int32_t* tile_m, int32_t* tile_n,
                                     int64_t* workgroups, int32_t* launches) {
  clear_error();
  if (plan == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan_info: plan is NULL");
  if (tile_m) *tile_m = plan->BM;
  if (tile_n) *tile_n = plan->BN;
  if (workgroups) *workgroups = plan->M == 0 ? 0 : plan->tiles_m * plan->tiles_n;
  if (launches)
    *launches = plan->M == 0 ? 0 : (plan->epi.reduction == FG_RED_LOGSUMEXP_ROW ? 2 : 1);
  return FG_OK;
}

extern "C" fg_status fgemm_run(const fg_plan* plan, const void* A, const void* W, const float* bias,
                               const float* gamma, const float* beta, void* out, void* workspace,
                               size_t ws_bytes, void* stream) {
  clear_error();
  if (plan == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_run: plan is NULL");
  const fg_plan& p = *plan;
  if (p.M == 0) return FG_OK;
  if (out == nullptr || (p.K > 0 && (A == nullptr || W == nullptr)))
    return fail(FG_ERR_INVALID_ARG, "fgemm_run: A, W (when K > 0) and out must be non-NULL");
  if (p.epi.has_bias && bias == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_run: bias is NULL");
  const int red = p.epi.reduction;
  if (red == FG_RED_GROUPNORM && (gamma == nullptr || beta == nullptr))
    return fail(FG_ERR_INVALID_ARG, "fgemm_run: GroupNorm needs gamma and beta");
  if (!aligned16(A) || !aligned16(W) || !aligned16(out))
    return fail(FG_ERR_ALIGNMENT, "fgemm_run: A, W and out must be 16-byte aligned");
  if (p.ws_bytes > 0) {
    if (workspace == nullptr || ws_bytes < p.ws_bytes)
      return fail(FG_ERR_WORKSPACE, "fgemm_run: workspace of %zu bytes needed, %zu given", p.ws_bytes,
                  workspace ? ws_bytes : (size_t)0);
    if (!aligned16(workspace)) return fail(FG_ERR_ALIGNMENT, "fgemm_run: workspace must be 16-byte aligned");
  }
  DenseArgs a;
  a.A = static_cast<const char*>(A);
  a.W = static_cast<const char*>(W);
  a.bias = p.epi.has_bias ? bias : nullptr;
  a.gamma = gamma;
  a.beta = beta;
  a.out = out;
  a.ws = static_cast<float2*>(workspace);
  a.M = (int)p.M;
  a.N = (int)p.N;
  a.K = p.K;
  a.tiles_n = (int)p.tiles_n;
  a.gn_width = red == FG_RED_GROUPNORM ? (int)(p.N / p.epi.gn_groups) : 0;
  a.gn_eps = p.epi.gn_eps;
  EpiArgs ep;
  memset(&ep, 0, sizeof(ep));
  ep.n_ops = p.epi.n_ops;
  for (int i = 0; i < p.epi.n_ops; ++i) {
    ep.kind[i] = p.epi.ops[i].kind;
    ep.a[i] = p.epi.ops[i].a;
    ep.b[i] = p.epi.ops[i].b;
  }
  const int out_k = p.out_dt == FG_BF16 ? OUT_BF16 : OUT_F32;
  KernelChoice kc{nullptr, 0};
  switch (p.cfg) {
    case CFG_F32: kc = pick_kernel<TileF32>(red, out_k); break;
    case CFG_BF16_256x128: kc = pick_kernel<TileBig>(red, out_k); break;
    case CFG_BF16_128x128: kc = pick_kernel<TileMid>(red, out_k); break;
  }
  if (kc.fn == nullptr) return fail(FG_ERR_UNSUPPORTED, "fgemm_run: no kernel for this plan");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const unsigned grid = (unsigned)(p.tiles_m * p.tiles_n);
  hipLaunchKernelGGL(kc.fn, dim3(grid), dim3(kc.threads), 0, s, a, ep);
  if (red == FG_RED_LOGSUMEXP_ROW) {
    const unsigned g2 = (unsigned)((p.M + 3) / 4);
    hipLaunchKernelGGL(lse_combine_kernel, dim3(g2), dim3(256), 0, s, a.ws, static_cast<float*>(out),
                       (int)p.M, (int)p.tiles_n);
  }
  return check_launch("fgemm_run");
}
