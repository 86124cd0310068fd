// fgemm.hip — the fused dense GEMM + tail: y = tail(x·Wᵀ + b).
//
// One kernel launch computes the GEMM on the matrix cores and applies the
// whole tail on the fp32 accumulators before its single store (paper §IV-B:
// layer-wise fusion, fp32 accumulation and post-processing). The one
// exception is a LogSumExp over a row that spans several N tiles: each tile
// writes its (max, Σexp) pair and a second launch of one wave per row
// combines them (the rescaling identity of online softmax, §I).
//
// When a problem has too few output tiles to occupy every compute unit with
// the large 256×256 tile, K is split into KS slices (split-K): every slice
// workgroup writes its fp32 partial tile to the workspace and counts its
// arrival on the tile's counter; the workgroup that arrives last adds the
// partials in slice order and runs the tail, so the tail still sees the
// complete accumulator and the result does not depend on arrival order.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
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
  const float* a_scale;   // e4m3: per-row scale of x [M]
  const float* w_scale;   // e4m3: per-row scale of W [N]
  void* out;
  float2* ws;
  int M, N;
  int64_t K;
  int tiles_m, tiles_n;
  int group_m;            // m-tiles per raster group (see tile_coords)
  int ks;                 // K slices (1 = no split)
  int64_t kslice;         // bytes of each row per slice but the last (multiple of 128)
  unsigned long long* counters;  // [tiles] (epoch << 32 | arrivals) words (split-K only)
  unsigned epoch;         // this run's epoch (split-K only)
  f32x4* partials;        // [tiles · ks · FM·FN · THREADS] partial tiles (split-K only)
  int gn_width;
  float gn_eps;
};

// Workgroup b runs on XCD b mod 8. When the launch is a multiple of 8, the
// tile order t = (b mod 8)·(G/8) + b/8 gives each XCD a contiguous range of
// t (slices fastest, then tile rows, then tile columns), so the slices of a
// tile share one L2 and so do the tiles that reuse the same W columns.
__device__ __forceinline__ int xcd_order(int b, int G) {
  return (G & 7) == 0 ? (b & 7) * (G >> 3) + (b >> 3) : b;
}

// Output tile of tile index `tile`: the tiles are walked in groups of GM
// tile rows, m fastest inside a group, so any run of consecutive indices —
// the tiles one XCD holds at a time — covers a block about GM rows tall and
// run/GM columns wide instead of a strip one or two columns wide. The L2 of
// that XCD then fetches GM row tiles of A and run/GM column tiles of W per
// K stage. The last group may be shorter.
__device__ __forceinline__ void tile_coords(int tile, int tiles_m, int tiles_n, int GM, int& tm, int& tn) {
  const int per_group = GM * tiles_n;
  const int g = tile / per_group, local = tile - g * per_group;
  const int rows = tiles_m - g * GM < GM ? tiles_m - g * GM : GM;
  tm = g * GM + local % rows;
  tn = local / rows;
}

// Split-K exchange (see slice_gather): the partial tiles of tile `tile` sit
// at partials + tile·ks·(one partial tile), its counter at counters[tile].
template <class TL>
__device__ __forceinline__ bool split_k_gather(const DenseArgs& a, int tile, int ks,
                                               f32x4 (&acc)[TL::FM][TL::FN], unsigned* flag) {
  constexpr int NF = TL::FM * TL::FN;
  return slice_gather<TL>(acc, a.partials + (size_t)tile * a.ks * NF * TL::THREADS, a.ks, ks, a.counters + tile,
                          a.epoch, flag);
}

template <class TL, int RED, int OUT>
__global__ __launch_bounds__(TL::THREADS) void fgemm_kernel(DenseArgs a, EpiArgs ep, EpiArgs post) {
  __shared__ __attribute__((aligned(16))) char lds[DenseLds<TL>::BYTES];
  const int t = xcd_order(blockIdx.x, a.tiles_m * a.tiles_n * a.ks);
  const int ks = t % a.ks, tile = t / a.ks;
  int tm, tn;
  tile_coords(tile, a.tiles_m, a.tiles_n, a.group_m, tm, tn);
  const int m0 = tm * TL::BM, n0 = tn * TL::BN;
  const int64_t rowbytes = a.K * TL::ESIZE;
  const int64_t kbeg = ks * a.kslice;
  const int64_t kbytes = ks == a.ks - 1 ? rowbytes - kbeg : a.kslice;

  BufRows<TL::A_LD, TL::RSTRIDE> ra;
  BufRows<TL::B_LD, TL::RSTRIDE> rb;
  ra.init(a.A + (int64_t)m0 * rowbytes + kbeg, a.M - m0, TL::BM, rowbytes);
  rb.init(a.W + (int64_t)n0 * rowbytes + kbeg, a.N - n0, TL::BN, rowbytes);

  // e4m3 (W8A8): the per-row scales of x and W, loaded before the K loop so
  // that their latency hides behind it
  float rsc[TL::IN == In::E4M3 ? TL::FM : 1][4], csc[TL::IN == In::E4M3 ? TL::FN : 1];
  if constexpr (TL::IN == In::E4M3) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + acc_row<TL>(fm, i);
        rsc[fm][i] = m < a.M ? a.a_scale[m] : 0.0f;
      }
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) {
      const int n = n0 + acc_col<TL>(fn);
      csc[fn] = n < a.N ? a.w_scale[n] : 0.0f;
    }
  }

  f32x4 acc[TL::FM][TL::FN];
  gemm_mainloop<TL>(ra, rb, kbytes, lds, acc, a.M - m0 < TL::BM ? a.M - m0 : TL::BM);
  if (a.ks > 1 && !split_k_gather<TL>(a, tile, ks, acc, reinterpret_cast<unsigned*>(lds))) return;

  if constexpr (TL::IN == In::E4M3) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[fm][fn][i] *= rsc[fm][i] * csc[fn];
  }
  if (a.bias != nullptr) add_bias<TL>(a.bias, n0, a.N, acc);
  apply_ops<TL>(ep, acc);

  float* red = reinterpret_cast<float*>(lds + DenseLds<TL>::MAIN);
  if constexpr (RED == FG_RED_LOGSUMEXP_ROW) {
    lse_partials<TL>(acc, red, m0, n0, a.M, a.N, tn, a.tiles_n, a.ws);
    return;
  }
  if constexpr (RED == FG_RED_GROUPNORM) {
    groupnorm_tile<TL>(acc, red, n0, a.N, a.gn_width, a.gn_eps, a.gamma, a.beta);
    apply_ops<TL>(post, acc);
  }

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

// out[m] = post(max_j m_j + log Σ_j s_j·exp(m_j − max_j m_j)); one wave per
// row.
__global__ __launch_bounds__(256) void lse_combine_kernel(const float2* ws, float* out, int M, int tiles_n,
                                                          EpiArgs post) {
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
  if (l == 0) {
    float v = mx + logf(s);
    for (int o = 0; o < post.n_ops; ++o) v = apply_op_scalar(post.kind[o], post.a[o], post.b[o], v);
    out[row] = v;
  }
}

// GroupNorm of groups that no tile holds in registers (wider than the tile,
// or not whole 16-column fragments): the GEMM launch has written the fp32
// pre-normalisation values z [M, N] (bias and ops applied) to the workspace,
// and this launch normalises them. One workgroup per row, one wave per group
// at a time: the group's mean, then its biased variance about the mean
// (each a wave-wide sum whose butterfly leaves the same value in every
// lane), then (z − μ)/√(σ² + eps)·γ + β, the post ops, and the store.
__global__ __launch_bounds__(256) void groupnorm_rows_kernel(const float* z, void* out, int out_bf16, int64_t N,
                                                             int gw, float eps, const float* gamma,
                                                             const float* beta, EpiArgs post) {
  const int64_t row = blockIdx.x;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const float* zr = z + row * N;
  const int groups = (int)(N / gw);
  const float inv_gw = 1.0f / (float)gw;
  for (int g = wave; g < groups; g += 4) {
    const float* zg = zr + (int64_t)g * gw;
    float s = 0.0f;
    for (int j = l; j < gw; j += 64) s += zg[j];
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) s += __shfl_xor(s, m, 64);
    const float mu = s * inv_gw;
    float q = 0.0f;
    for (int j = l; j < gw; j += 64) {
      const float d = zg[j] - mu;
      q += d * d;
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) q += __shfl_xor(q, m, 64);
    const float rstd = fast_rsqrt(q * inv_gw + eps);
    for (int j = l; j < gw; j += 64) {
      const int64_t n = (int64_t)g * gw + j;
      float v = (zg[j] - mu) * rstd * gamma[n] + beta[n];
      for (int o = 0; o < post.n_ops; ++o) v = apply_op_scalar(post.kind[o], post.a[o], post.b[o], v);
      if (out_bf16)
        static_cast<uint16_t*>(out)[row * N + n] = f32_to_bf16_bits(v);
      else
        static_cast<float*>(out)[row * N + n] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// kernel table

typedef Tile<In::F32, 64, 128> TileF32;
typedef Tile<In::BF16, 256, 256, 2, 4> TileHuge;
typedef Tile<In::BF16, 256, 128, 4, 2> TileBig;
typedef Tile<In::BF16, 128, 128> TileMid;
typedef Tile<In::E4M3, 256, 128, 4, 2> TileF8Big;
typedef Tile<In::E4M3, 128, 128> TileF8Mid;

enum Cfg : int {
  CFG_F32 = 0,
  CFG_BF16_256x128 = 1,
  CFG_BF16_128x128 = 2,
  CFG_BF16_256x256 = 3,
  CFG_E4M3_256x128 = 4,
  CFG_E4M3_128x128 = 5
};

// Relative MFMA efficiency of the bf16 tiles, measured on 1024..4096-row
// problems: the larger tile moves fewer bytes from L2 into LDS per FLOP.
struct TileModel {
  int cfg, BM, BN;
  double eff;
};

// Tile width and wave tile width of each configuration (host copies of the
// Tile parameters above), and the host twin of groupnorm_fits_tile.
static void cfg_widths(int cfg, int& BN, int& TN) {
  switch (cfg) {
    case CFG_F32: BN = TileF32::BN; TN = TileF32::TN; break;
    case CFG_BF16_256x256: BN = TileHuge::BN; TN = TileHuge::TN; break;
    case CFG_BF16_256x128: BN = TileBig::BN; TN = TileBig::TN; break;
    case CFG_BF16_128x128: BN = TileMid::BN; TN = TileMid::TN; break;
    case CFG_E4M3_256x128: BN = TileF8Big::BN; TN = TileF8Big::TN; break;
    default: BN = TileF8Mid::BN; TN = TileF8Mid::TN; break;
  }
}
static bool groupnorm_in_tile(int cfg, int64_t gw) {
  int BN, TN;
  cfg_widths(cfg, BN, TN);
  return gw % 16 == 0 && (gw <= TN ? TN % gw == 0 : (gw % TN == 0 && BN % gw == 0));
}
static const TileModel kBf16Tiles[] = {
    {CFG_BF16_256x256, 256, 256, 1.00},
    {CFG_BF16_256x128, 256, 128, 0.88},
    {CFG_BF16_128x128, 128, 128, 0.72},
};
// e4m3 tiles (W8A8): relative efficiencies measured on the 1024-row shape.
static const TileModel kE4m3Tiles[] = {
    {CFG_E4M3_256x128, 256, 128, 0.88},
    {CFG_E4M3_128x128, 128, 128, 0.72},
};

typedef void (*KernelFn)(DenseArgs, EpiArgs, EpiArgs);

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
  int ks;                   // K slices
  int64_t kslice;           // bytes per row per slice (all but the last)
  int64_t tiles_m, tiles_n;
  size_t lse_bytes;         // LogSumExp pairs at the start of the workspace
  int gn_two_pass;          // GroupNorm groups no tile holds: fp32 z in the workspace, second launch
  size_t z_bytes;           // that z [M, N] at the start of the workspace
  size_t cnt_off, part_off; // split-K counters and partial tiles
  size_t ws_bytes;
};

static size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }



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
  if (in_dtype != FG_F32 && in_dtype != FG_BF16 && in_dtype != FG_E4M3)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: input dtype %d not supported (f32, bf16 or e4m3)", in_dtype);
  if (out_dtype != FG_F32 && out_dtype != FG_BF16)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: output dtype %d not supported (f32 or bf16)", out_dtype);
  if (epi->n_ops < 0 || epi->n_ops > FG_MAX_OPS)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: n_ops=%d outside 0..%d", epi->n_ops, FG_MAX_OPS);
  if (epi->n_post_ops < 0 || epi->n_post_ops > FG_MAX_OPS)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: n_post_ops=%d outside 0..%d", epi->n_post_ops, FG_MAX_OPS);
  for (int chain = 0; chain < 2; ++chain) {
    const fg_op* ops = chain == 0 ? epi->ops : epi->post_ops;
    const int n = chain == 0 ? epi->n_ops : epi->n_post_ops;
    const char* what = chain == 0 ? "op" : "post op";
    for (int i = 0; i < n; ++i) {
      const fg_op& op = ops[i];
      if (op.kind < FG_OP_SCALE || op.kind > FG_OP_LEAKY_RELU)
        return fail(FG_ERR_INVALID_ARG, "fgemm_plan: %s %d has unknown kind %d", what, i, op.kind);
      if (op.kind == FG_OP_CLAMP && !(op.a <= op.b))
        return fail(FG_ERR_INVALID_ARG, "fgemm_plan: clamp %s %d needs lo <= hi", what, i);
      if (!isfinite(op.a) || !isfinite(op.b))
        return fail(FG_ERR_INVALID_ARG, "fgemm_plan: %s %d has a non-finite parameter", what, i);
    }
  }
  if (epi->has_bias != 0 && epi->has_bias != 1)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: has_bias must be 0 or 1");
  const int red = epi->reduction;
  if (red != FG_RED_NONE && red != FG_RED_LOGSUMEXP_ROW && red != FG_RED_GROUPNORM)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: unknown reduction %d", red);
  if (red == FG_RED_NONE && epi->n_post_ops != 0)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: post ops need a reduction (append them to ops instead)");
  if (red == FG_RED_LOGSUMEXP_ROW && out_dtype != FG_F32)
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: LogSumExp output must be f32");
  const int64_t esize = in_dtype == FG_F32 ? 4 : in_dtype == FG_BF16 ? 2 : 1;
  const int epc = (int)(16 / esize);
  if (K % epc != 0)
    return fail(FG_ERR_ALIGNMENT, "fgemm_plan: K=%lld must be a multiple of %d", (long long)K, epc);
  // tile operands are addressed with 32-bit offsets from the tile's first row
  if (K * esize > (int64_t)(1 << 22))
    return fail(FG_ERR_UNSUPPORTED, "fgemm_plan: K=%lld exceeds the 4 MiB row limit", (long long)K);
  if (red != FG_RED_LOGSUMEXP_ROW) {
    const int opc = out_dtype == FG_F32 ? 4 : 8;
    if (N % opc != 0)
      return fail(FG_ERR_ALIGNMENT, "fgemm_plan: N=%lld must be a multiple of %d", (long long)N, opc);
  }
  int64_t gw = 0;
  if (red == FG_RED_GROUPNORM) {
    if (epi->gn_groups <= 0 || N % epi->gn_groups != 0)
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: N=%lld not divisible into %d groups", (long long)N,
                  epi->gn_groups);
    if (!(epi->gn_eps >= 0.0f) || !isfinite(epi->gn_eps))
      return fail(FG_ERR_INVALID_ARG, "fgemm_plan: gn_eps must be finite and >= 0");
    gw = N / epi->gn_groups;
  }

  fg_plan* p = new (std::nothrow) fg_plan();
  if (p == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan: out of host memory");
  p->M = M;
  p->N = N;
  p->K = K;
  p->in_dt = in_dtype;
  p->out_dt = out_dtype;
  p->epi = *epi;
  p->ks = 1;
  if (in_dtype == FG_F32) {
    p->cfg = CFG_F32;
    p->BM = TileF32::BM;
    p->BN = TileF32::BN;
  } else if (in_dtype == FG_E4M3) {
    // W8A8: the tile that minimises workgroups per compute unit × tile work
    // / tile efficiency; no K split
    double best = 0.0;
    for (const TileModel& tmod : kE4m3Tiles) {
      const int64_t tiles = ((M + tmod.BM - 1) / tmod.BM) * ((N + tmod.BN - 1) / tmod.BN);
      const double cost = (double)((tiles + 255) / 256) * tmod.BM * tmod.BN / tmod.eff;
      if (best == 0.0 || cost < best) {
        best = cost;
        p->cfg = tmod.cfg;
        p->BM = tmod.BM;
        p->BN = tmod.BN;
      }
    }
  } else {
    // Estimated time of each (tile, K slices) choice: the workgroups one of
    // the 256 compute units runs × work per workgroup / tile efficiency, with
    // 3 % per extra slice for the partial-tile exchange. K is split only
    // when the 256×256 tiles would leave at least three quarters of the
    // compute units idle: a split concentrates the tail of each tile on one
    // workgroup and adds the partial-tile exchange, which costs more than it
    // gains once the tiles already cover much of the chip. Slices stay
    // powers of two and at least 16 stages of 64 K-values each.
    double best = 0.0;
    for (const TileModel& tmod : kBf16Tiles) {
      const int64_t tiles = ((M + tmod.BM - 1) / tmod.BM) * ((N + tmod.BN - 1) / tmod.BN);
      for (int ks = 1; ks <= 4; ks *= 2) {
        if (ks > 1 && (tmod.cfg != CFG_BF16_256x256 || tiles > 64 || K / 64 < 16 * ks)) break;
        const int64_t per_cu = (tiles * ks + 255) / 256;
        const double cost = (double)per_cu * tmod.BM * tmod.BN * ((double)K / ks + 64.0) / tmod.eff *
                            (1.0 + 0.03 * (ks - 1));
        if (best == 0.0 || cost < best) {
          best = cost;
          p->cfg = tmod.cfg;
          p->BM = tmod.BM;
          p->BN = tmod.BN;
          p->ks = ks;
        }
      }
    }
  }
  // GroupNorm: widths of 256 channels need the 256-column tile; groups no
  // tile holds in registers take the second launch
  p->gn_two_pass = 0;
  if (red == FG_RED_GROUPNORM && !groupnorm_in_tile(p->cfg, gw)) {
    if (in_dtype == FG_BF16 && groupnorm_in_tile(CFG_BF16_256x256, gw)) {
      p->cfg = CFG_BF16_256x256;
      p->BM = TileHuge::BM;
      p->BN = TileHuge::BN;
    } else {
      p->gn_two_pass = 1;
    }
  }
  p->tiles_m = (M + p->BM - 1) / p->BM;
  p->tiles_n = (N + p->BN - 1) / p->BN;
  if (p->tiles_m * p->tiles_n > LIM) {
    delete p;
    return fail(FG_ERR_INVALID_ARG, "fgemm_plan: too many tiles");
  }
  const int64_t stages = K * esize / 128;
  p->kslice = p->ks > 1 ? (stages / p->ks) * 128 : 0;
  p->lse_bytes = red == FG_RED_LOGSUMEXP_ROW ? (size_t)M * (size_t)p->tiles_n * sizeof(float2) : 0;
  p->z_bytes = p->gn_two_pass ? (size_t)M * (size_t)N * sizeof(float) : 0;
  if (p->z_bytes > 0) p->lse_bytes = p->z_bytes;   // the workspace's first region holds z instead
  p->cnt_off = round256(p->lse_bytes);
  p->part_off = p->cnt_off;
  p->ws_bytes = p->lse_bytes;
  if (p->ks > 1) {
    const size_t tiles = (size_t)(p->tiles_m * p->tiles_n);
    p->part_off = round256(p->cnt_off + tiles * sizeof(unsigned long long));
    p->ws_bytes = p->part_off + tiles * (size_t)p->ks * (size_t)p->BM * (size_t)p->BN * sizeof(float);
  }
  *plan = p;
  return FG_OK;
}

extern "C" size_t fgemm_workspace_bytes(const fg_plan* plan) { return plan ? plan->ws_bytes : 0; }

extern "C" void fgemm_destroy(fg_plan* plan) { delete plan; }

extern "C" fg_status fgemm_plan_info(const fg_plan* plan, int32_t* tile_m, int32_t* tile_n,
                                     int64_t* workgroups, int32_t* launches, int32_t* k_slices) {
  clear_error();
  if (plan == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_plan_info: plan is NULL");
  if (tile_m) *tile_m = plan->BM;
  if (tile_n) *tile_n = plan->BN;
  if (workgroups) *workgroups = plan->M == 0 ? 0 : plan->tiles_m * plan->tiles_n * plan->ks;
  if (launches)
    *launches = plan->M == 0 ? 0 : (plan->epi.reduction == FG_RED_LOGSUMEXP_ROW || plan->gn_two_pass ? 2 : 1);
  if (k_slices) *k_slices = plan->ks;
  return FG_OK;
}

static fg_status run_plan(const fg_plan* plan, const void* A, const void* W, const float* a_scale,
                          const float* w_scale, const float* bias, const float* gamma, const float* beta, void* out,
                          void* workspace, size_t ws_bytes, void* stream) {
  if (plan == nullptr) return fail(FG_ERR_INVALID_ARG, "fgemm_run: plan is NULL");
  const fg_plan& p = *plan;
  if (p.M == 0) return FG_OK;
  if (p.in_dt == FG_E4M3 && (a_scale == nullptr || w_scale == nullptr))
    return fail(FG_ERR_INVALID_ARG, "fgemm_run: an e4m3 plan needs per-row scales (fgemm_run_scaled)");
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
  a.a_scale = a_scale;
  a.w_scale = w_scale;
  a.out = out;
  a.ws = static_cast<float2*>(workspace);
  a.M = (int)p.M;
  a.N = (int)p.N;
  a.K = p.K;
  a.tiles_m = (int)p.tiles_m;
  a.group_m = (int)(p.tiles_m < 4 ? p.tiles_m : 4);
  a.tiles_n = (int)p.tiles_n;
  a.ks = p.ks;
  a.kslice = p.kslice;
  a.counters = p.ks > 1 ? reinterpret_cast<unsigned long long*>(static_cast<char*>(workspace) + p.cnt_off) : nullptr;
  a.epoch = p.ks > 1 ? next_epoch() : 0;
  a.partials = p.ks > 1 ? reinterpret_cast<f32x4*>(static_cast<char*>(workspace) + p.part_off) : nullptr;
  a.gn_width = red == FG_RED_GROUPNORM ? (int)(p.N / p.epi.gn_groups) : 0;
  a.gn_eps = p.epi.gn_eps;
  EpiArgs ep, post;
  memset(&ep, 0, sizeof(ep));
  memset(&post, 0, sizeof(post));
  ep.n_ops = p.epi.n_ops;
  for (int i = 0; i < p.epi.n_ops; ++i) {
    ep.kind[i] = p.epi.ops[i].kind;
    ep.a[i] = p.epi.ops[i].a;
    ep.b[i] = p.epi.ops[i].b;
  }
  post.n_ops = p.epi.n_post_ops;
  for (int i = 0; i < p.epi.n_post_ops; ++i) {
    post.kind[i] = p.epi.post_ops[i].kind;
    post.a[i] = p.epi.post_ops[i].a;
    post.b[i] = p.epi.post_ops[i].b;
  }
  // two-pass GroupNorm: the GEMM launch writes fp32 z (bias and ops
  // applied) to the workspace as a plain fp32 output
  const int kred = p.gn_two_pass ? FG_RED_NONE : red;
  const int out_k = p.gn_two_pass ? OUT_F32 : (p.out_dt == FG_BF16 ? OUT_BF16 : OUT_F32);
  if (p.gn_two_pass) a.out = workspace;
  KernelChoice kc{nullptr, 0};
  switch (p.cfg) {
    case CFG_F32: kc = pick_kernel<TileF32>(kred, out_k); break;
    case CFG_BF16_256x256: kc = pick_kernel<TileHuge>(kred, out_k); break;
    case CFG_BF16_256x128: kc = pick_kernel<TileBig>(kred, out_k); break;
    case CFG_BF16_128x128: kc = pick_kernel<TileMid>(kred, out_k); break;
    case CFG_E4M3_256x128: kc = pick_kernel<TileF8Big>(kred, out_k); break;
    case CFG_E4M3_128x128: kc = pick_kernel<TileF8Mid>(kred, out_k); break;
  }
  if (kc.fn == nullptr) return fail(FG_ERR_UNSUPPORTED, "fgemm_run: no kernel for this plan");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const unsigned grid = (unsigned)(p.tiles_m * p.tiles_n * p.ks);
  Launches lc;
  lc.add(launch(kc.fn, dim3(grid), dim3(kc.threads), 0, s, a, ep, post));
  if (p.gn_two_pass)
    lc.add(launch(groupnorm_rows_kernel, dim3((unsigned)p.M), dim3(256), 0, s,
                  static_cast<const float*>(workspace), out, p.out_dt == FG_BF16 ? 1 : 0, p.N,
                  (int)(p.N / p.epi.gn_groups), p.epi.gn_eps, gamma, beta, post));
  if (red == FG_RED_LOGSUMEXP_ROW) {
    const unsigned g2 = (unsigned)((p.M + 3) / 4);
    lc.add(launch(lse_combine_kernel, dim3(g2), dim3(256), 0, s, a.ws, static_cast<float*>(out), (int)p.M,
                  (int)p.tiles_n, post));
  }
  return check_launch("fgemm_run", lc);
}

extern "C" fg_status fgemm_run(const fg_plan* plan, const void* A, const void* W, const float* bias,
                               const float* gamma, const float* beta, void* out, void* workspace,
                               size_t ws_bytes, void* stream) {
  clear_error();
  return run_plan(plan, A, W, nullptr, nullptr, bias, gamma, beta, out, workspace, ws_bytes, stream);
}

extern "C" fg_status fgemm_run_scaled(const fg_plan* plan, const void* A, const void* W, const float* a_scale,
                                      const float* w_scale, const float* bias, const float* gamma,
                                      const float* beta, void* out, void* workspace, size_t ws_bytes,
                                      void* stream) {
  clear_error();
  return run_plan(plan, A, W, a_scale, w_scale, bias, gamma, beta, out, workspace, ws_bytes, stream);
}
