// moe.hip — one MoE expert-FFN step of a gpt-oss-20b-like layer.
//
// Launch sequence on the caller's stream, with no host synchronisation (the
// per-expert counts never leave the device):
//   [e4m3 only] quantise tokens per row          quantize_rows_kernel
//   route: top-k + softmax per token             moe_route_kernel
//   histogram, offsets, stable permutation       moe_permute_kernel (one workgroup)
//   grouped gate/up GEMM + clamped SwiGLU        grouped_kernel<.., EPI_GATEUP>
//   [e4m3 only] quantise h per row               quantize_rows_kernel
//   grouped down GEMM × routing weight           grouped_kernel<.., EPI_DOWN>
//   finalize: Σ_j over the k slots of a token     moe_finalize_kernel
// The token gather is folded into the gate/up GEMM's A-row addresses, and
// the scatter back to slot order into the down GEMM's store addresses, so no
// permuted copy of the tokens or of the outputs is ever materialised.
//
// Paper §IV-A optimises this block's decode kernels (MoE finalize, Table I);
// §V names optimising the whole MoE-MLP block jointly as the next step.
#include <hip/hip_runtime.h>
#include <math.h>

#include "fg_host.hpp"
#include "fg_quant.hpp"
#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

__global__ void quantize_rows_kernel(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, float* s);

constexpr int KMAX = 8;       // largest supported top_k
constexpr int EMAX = 256;     // largest supported expert count

// ---------------------------------------------------------------------------
// route: per token, the top-k logits in descending order with ties to the
// lower expert index, then the softmax over them. The list is kept sorted by
// the key (value descending, index ascending) with an insertion pass that
// compares full keys, so an entry displaced downwards still lands ahead of
// equal values with larger indices.

__global__ __launch_bounds__(256) void moe_route_kernel(const float* logits, int T, int E, int k,
                                                        int32_t* topk_idx, float* topk_w) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  float bv[KMAX];
  int bi[KMAX];
#pragma unroll
  for (int p = 0; p < KMAX; ++p) {
    bv[p] = -INFINITY;
    bi[p] = -1;
  }
  const float* row = logits + (int64_t)t * E;
  for (int e = 0; e < E; ++e) {
    float v = row[e];
    int id = e;
#pragma unroll
    for (int p = 0; p < KMAX; ++p) {
      // branch-free compare-exchange on the key (value desc, index asc); an
      // empty slot (index −1) always takes the carried entry
      const bool take = (bi[p] < 0) | (v > bv[p]) | ((v == bv[p]) & (id < bi[p]));
      const float nv = take ? v : bv[p];
      const int ni = take ? id : bi[p];
      v = take ? bv[p] : v;
      id = take ? bi[p] : id;
      bv[p] = nv;
      bi[p] = ni;
    }
  }
  float ex[KMAX], sum = 0.0f;
#pragma unroll
  for (int p = 0; p < KMAX; ++p) {
    ex[p] = p < k ? expf(bv[p] - bv[0]) : 0.0f;
    sum += ex[p];
  }
#pragma unroll
  for (int p = 0; p < KMAX; ++p) {
    if (p < k) {
      topk_idx[(int64_t)t * k + p] = bi[p];
      topk_w[(int64_t)t * k + p] = ex[p] / sum;
    }
  }
}

// ---------------------------------------------------------------------------
// permute: one workgroup of 16 waves. Wave w owns experts w, w + 16, ...; it
// walks the S = T·k slot ids in 64-slot chunks and, with one ballot per
// chunk, counts (pass 1) and then places (pass 2) the slots of its expert:
// a slot's position is the expert's offset plus the number of its expert's
// slots with a smaller id. That is the stable sort by (expert, slot id),
// computed without atomics, so it is unique and bit-reproducible.

constexpr int PERM_THREADS = 1024;
constexpr int PERM_LDS_SLOTS = 65536;

template <bool IDS_IN_LDS>
__global__ __launch_bounds__(PERM_THREADS) void moe_permute_kernel(const int32_t* topk_idx, int S, int E, int BM,
                                                                   int32_t* offsets, int32_t* tile_off,
                                                                   int32_t* perm) {
  __shared__ int cnt[EMAX];
  __shared__ int off[EMAX + 1];
  __shared__ uint8_t ids_lds[IDS_IN_LDS ? PERM_LDS_SLOTS : 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if constexpr (IDS_IN_LDS) {
    for (int i = tid; i < S; i += PERM_THREADS) ids_lds[i] = (uint8_t)topk_idx[i];
    __syncthreads();
  }
  auto expert_of = [&](int s) -> int {
    if constexpr (IDS_IN_LDS) return ids_lds[s];
    else return topk_idx[s];
  };
  for (int e = wave; e < E; e += PERM_THREADS / 64) {
    int c = 0;
    for (int base = 0; base < S; base += 64) {
      const int s = base + lane;
      const bool m = s < S && expert_of(s) == e;
      c += __popcll(__ballot(m));
    }
    if (lane == 0) cnt[e] = c;
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0, tacc = 0;
    for (int e = 0; e < E; ++e) {
      off[e] = acc;
      offsets[e] = acc;
      tile_off[e] = tacc;
      acc += cnt[e];
      tacc += (cnt[e] + BM - 1) / BM;
    }
    off[E] = acc;
    offsets[E] = acc;
    tile_off[E] = tacc;
  }
  __syncthreads();
  for (int e = wave; e < E; e += PERM_THREADS / 64) {
    int run = off[e];
    for (int base = 0; base < S; base += 64) {
      const int s = base + lane;
      const bool m = s < S && expert_of(s) == e;
      const unsigned long long mask = __ballot(m);
      if (m) {
        const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                    __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
        perm[run + below] = s;
      }
      run += __popcll(mask);
    }
  }
}

// ---------------------------------------------------------------------------
// grouped GEMMs. The launch covers an upper bound of m-tiles,
// Σ_e ceil(n_e/BM) ≤ S/BM + E; workgroup id → (global m-tile, n-tile), and the
// global m-tile → expert by binary search of the device-side tile prefix
// written by the permute kernel. Workgroups past the last tile exit at once.

enum : int { EPI_GATEUP = 0, EPI_DOWN = 1 };

struct GroupedArgs {
  const char* A;           // gate/up: tokens [T, H] (bf16 or e4m3); down: h [S, I]
  const char* W;           // [E, Nw, K] expert weights (bf16 or e4m3)
  const float* a_scale;    // e4m3: per-row activation scale (gate/up: per token; down: per slot row)
  const float* w_scale;    // e4m3: [E, Nw] per-row weight scale
  const int32_t* perm;     // [S] slot ids in expert order
  const int32_t* offsets;  // [E + 1]
  const int32_t* tile_off; // [E + 1]
  const float* topk_w;     // [S] routing weights by slot id
  char* out;               // gate/up: h [S, I] bf16 (expert order); down: y_slot [S, H] bf16 (slot order)
  int E, k, tiles_n;
  int64_t K;               // contraction length in elements
  int64_t Nw;              // weight rows per expert: 2I or H
  int64_t I;               // intermediate size (gate/up pairing)
  int64_t ldo;             // output row length in elements
  float alpha, limit;
  int interleaved;
};

template <class TL>
struct GroupedLds {
  static constexpr int OUT_STAGE = TL::BM * (TL::BN * 2 + 16);
  static constexpr int BYTES = TL::LOOP_LDS > OUT_STAGE ? TL::LOOP_LDS : OUT_STAGE;
};

// Weight row of tile-local B row ρ. Gate/up tiles interleave 16-row blocks:
// block f (ρ/16) is gate (f even) or up (f odd) of output columns
// (f/2)·16 .. +15, so a lane's accumulators for fragment pairs (2q, 2q+1)
// hold matching gate and up values.
template <class TL, int EPI>
__device__ __forceinline__ int64_t weight_row(const GroupedArgs& a, int tn, int rho) {
  if constexpr (EPI == EPI_GATEUP) {
    const int f = rho >> 4;
    const int64_t hc = (int64_t)tn * (TL::BN / 2) + (f >> 1) * 16 + (rho & 15);
    const int up = f & 1;
    return a.interleaved ? 2 * hc + up : up * a.I + hc;
  } else {
    const int64_t n = (int64_t)tn * TL::BN + rho;
    return n < a.Nw ? n : a.Nw - 1;
  }
}

template <class TL, int EPI>
__global__ __launch_bounds__(TL::THREADS) void grouped_kernel(GroupedArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[GroupedLds<TL>::BYTES];
  const int tn = blockIdx.x % a.tiles_n;
  const int mt = blockIdx.x / a.tiles_n;
  if (mt >= a.tile_off[a.E]) return;
  int lo = 0, hi = a.E;        // tile_off[lo] ≤ mt < tile_off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.tile_off[mid] <= mt) lo = mid;
    else hi = mid;
  }
  const int e = lo;
  const int seg0 = a.offsets[e], seg1 = a.offsets[e + 1];
  const int r0 = seg0 + (mt - a.tile_off[e]) * TL::BM;
  const int64_t rowbytes = a.K * TL::ESIZE;
  const int tr = threadIdx.x >> 3;

  RowSet<TL::A_LD> ra;
  RowSet<TL::B_LD> rb;
#pragma unroll
  for (int p = 0; p < TL::A_LD; ++p) {
    int r = r0 + tr + TL::RSTRIDE * p;
    r = r < seg1 ? r : seg0;
    const int64_t arow = EPI == EPI_GATEUP ? (int64_t)(a.perm[r] / a.k) : (int64_t)r;
    ra.ptr[p] = a.A + arow * rowbytes;
  }
  const char* We = a.W + (int64_t)e * a.Nw * rowbytes;
#pragma unroll
  for (int p = 0; p < TL::B_LD; ++p) rb.ptr[p] = We + weight_row<TL, EPI>(a, tn, tr + TL::RSTRIDE * p) * rowbytes;

  f32x4 acc[TL::FM][TL::FN];
  gemm_mainloop<TL>(ra, rb, rowbytes, lds, acc);

  const int l = threadIdx.x & 63, wave = threadIdx.x >> 6, wn = wave % TL::WN;
  // per accumulator row: the scale of its activation row (e4m3) and, for the
  // down GEMM, the routing weight of its slot
  float rs[TL::FM][4];
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = r0 + acc_row<TL>(fm, i);
      r = r < seg1 ? r : seg0;
      float s = 1.0f;
      if constexpr (TL::IN == In::E4M3)
        s = EPI == EPI_GATEUP ? a.a_scale[a.perm[r] / a.k] : a.a_scale[r];
      if constexpr (EPI == EPI_DOWN) s *= a.topk_w[a.perm[r]];
      rs[fm][i] = s;
    }
  float ws[TL::FN];
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    ws[fn] = 1.0f;
    if constexpr (TL::IN == In::E4M3)
      ws[fn] = a.w_scale[(int64_t)e * a.Nw + weight_row<TL, EPI>(a, tn, acc_col<TL>(fn))];
  }
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[fm][fn][i] *= rs[fm][i] * ws[fn];

  if constexpr (EPI == EPI_GATEUP) {
    const float alpha = a.alpha, limit = a.limit;
    char* out = a.out;
    const int64_t ldo = a.ldo;
    const int c0 = tn * (TL::BN / 2);
    store_tile_bf16<TL, TL::BN / 2>(
        lds,
        [&](int fm, int fn, int i, float& v, int& c) {
          if (fn & 1) return false;
          // clamped SwiGLU: g = min(gate, L), u = clamp(up, −L, L), (u + 1)·g·σ(αg)
          const float g = fminf(acc[fm][fn][i], limit);
          const float u = fminf(fmaxf(acc[fm][fn + 1][i], -limit), limit);
          v = (u + 1.0f) * (g / (1.0f + expf(-alpha * g)));
          c = ((wn * TL::FN + fn) >> 1) * 16 + (l & 15);
          return true;
        },
        [&](int r) -> char* {
          const int row = r0 + r;
          return row < seg1 ? out + ((int64_t)row * ldo + c0) * 2 : nullptr;
        },
        TL::BN / 2);
  } else {
    char* out = a.out;
    const int64_t ldo = a.ldo;
    const int n0 = tn * TL::BN;
    const int ncols = (int)(a.Nw - n0 < TL::BN ? a.Nw - n0 : TL::BN);
    store_tile_bf16<TL, TL::BN>(
        lds,
        [&](int fm, int fn, int i, float& v, int& c) {
          v = acc[fm][fn][i];
          c = acc_col<TL>(fn);
          return true;
        },
        [&](int r) -> char* {
          const int row = r0 + r;
          return row < seg1 ? out + ((int64_t)a.perm[row] * ldo + n0) * 2 : nullptr;
        },
        ncols);
  }
}

// ---------------------------------------------------------------------------
// finalize: out[t, :] = Σ_j y_slot[t·k + j, :], j ascending, fp32 sum, bf16 out.
// One thread per 8 consecutive columns of a token.

__global__ __launch_bounds__(256) void moe_finalize_kernel(const uint16_t* y_slot, uint16_t* out, int T,
                                                           int64_t H, int k) {
  const int64_t cpt = H / 8;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = idx / cpt, c = idx % cpt;
  if (t >= T) return;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int j = 0; j < k; ++j) {
    const i32x4 v = *reinterpret_cast<const i32x4*>(y_slot + ((t * k + j) * H + c * 8));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc[2 * q] += bf16_bits_to_f32((uint16_t)(v[q] & 0xffff));
      acc[2 * q + 1] += bf16_bits_to_f32((uint16_t)((uint32_t)v[q] >> 16));
    }
  }
  i32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = (int)((uint32_t)f32_to_bf16_bits(acc[2 * q]) | ((uint32_t)f32_to_bf16_bits(acc[2 * q + 1]) << 16));
  *reinterpret_cast<i32x4*>(out + (t * H + c * 8)) = o;
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---------------------------------------------------------------------------
// host side

typedef Tile<In::BF16, 128, 128> GBf16Big;
typedef Tile<In::BF16, 32, 128> GBf16Small;
typedef Tile<In::E4M3, 128, 128> GF8Big;
typedef Tile<In::E4M3, 32, 128> GF8Small;

struct MoeLayout {
  int64_t S;
  int BM;
  size_t tile_off, h, y, xq, sx, hq, sh, total;
};

static size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

// Row tile of the grouped GEMMs: 128 rows when experts average more than 48
// slots, else 32 (decode: a handful of rows per expert, weight streaming).
static int pick_bm(int64_t S, int E) { return S > (int64_t)48 * E ? 128 : 32; }

static MoeLayout layout(const moe_desc& d) {
  MoeLayout L;
  L.S = d.T * d.top_k;
  L.BM = pick_bm(L.S, d.E);
  size_t o = 0;
  L.tile_off = o;
  o = align_up(o + sizeof(int32_t) * (size_t)(d.E + 1));
  L.h = o;
  o = align_up(o + (size_t)L.S * (size_t)d.I * 2);
  L.y = o;
  o = align_up(o + (size_t)L.S * (size_t)d.H * 2);
  L.xq = L.sx = L.hq = L.sh = 0;
  if (d.w_dtype == FG_E4M3) {
    L.xq = o;
    o = align_up(o + (size_t)d.T * (size_t)d.H);
    L.sx = o;
    o = align_up(o + sizeof(float) * (size_t)d.T);
    L.hq = o;
    o = align_up(o + (size_t)L.S * (size_t)d.I);
    L.sh = o;
    o = align_up(o + sizeof(float) * (size_t)L.S);
  }
  L.total = o;
  return L;
}

static fg_status validate_desc(const moe_desc* d, const char* fn) {
  if (d == nullptr) return fail(FG_ERR_INVALID_ARG, "%s: desc is NULL", fn);
  if (d->T < 0 || d->T > 0x7fffffffLL) return fail(FG_ERR_INVALID_ARG, "%s: bad T=%lld", fn, (long long)d->T);
  if (d->H <= 0 || d->I <= 0 || d->H > (1 << 20) || d->I > (1 << 20))
    return fail(FG_ERR_INVALID_ARG, "%s: bad H=%lld or I=%lld", fn, (long long)d->H, (long long)d->I);
  if (d->H % 64 != 0 || d->I % 64 != 0)
    return fail(FG_ERR_ALIGNMENT, "%s: H and I must be multiples of 64", fn);
  if (d->E < 1 || d->E > EMAX) return fail(FG_ERR_INVALID_ARG, "%s: E=%d outside 1..%d", fn, d->E, EMAX);
  if (d->top_k < 1 || d->top_k > KMAX || d->top_k > d->E)
    return fail(FG_ERR_INVALID_ARG, "%s: top_k=%d outside 1..min(E, %d)", fn, d->top_k, KMAX);
  if (d->T * d->top_k > 0x7fffffffLL) return fail(FG_ERR_INVALID_ARG, "%s: T*top_k too large", fn);
  if (d->w_dtype != FG_BF16 && d->w_dtype != FG_E4M3)
    return fail(d->w_dtype == FG_F32 ? FG_ERR_UNSUPPORTED : FG_ERR_INVALID_ARG,
                "%s: w_dtype %d not supported (bf16 or e4m3)", fn, d->w_dtype);
  if (!isfinite(d->swiglu_alpha) || !isfinite(d->swiglu_limit) || !(d->swiglu_limit >= 0.0f))
    return fail(FG_ERR_INVALID_ARG, "%s: swiglu_alpha must be finite and swiglu_limit finite and >= 0", fn);
  if (d->gateup_interleaved != 0 && d->gateup_interleaved != 1)
    return fail(FG_ERR_INVALID_ARG, "%s: gateup_interleaved must be 0 or 1", fn);
  return FG_OK;
}

template <class TL, int EPI>
static void launch_grouped(const GroupedArgs& a, int64_t S, hipStream_t s) {
  const int64_t mtiles = (S + (int64_t)a.E * (TL::BM - 1)) / TL::BM;
  const unsigned grid = (unsigned)(mtiles * a.tiles_n);
  hipLaunchKernelGGL((grouped_kernel<TL, EPI>), dim3(grid), dim3(TL::THREADS), 0, s, a);
}

}  // namespace fg

using namespace fg;

extern "C" size_t moe_workspace_bytes(const moe_desc* d) {
  if (validate_desc(d, "moe_workspace_bytes") != FG_OK) return 0;
  return layout(*d).total;
}

extern "C" fg_status moe_grouped_ffn(const moe_desc* d, const void* tokens, const float* router_logits,
                                     const void* w_gateup, const void* w_down, const float* s_gateup,
                                     const float* s_down, void* out, int32_t* topk_idx, float* topk_w,
                                     int32_t* perm, int32_t* expert_offsets, void* workspace, size_t ws_bytes,
                                     void* stream) {
  clear_error();
  const char* fn = "moe_grouped_ffn";
  fg_status st = validate_desc(d, fn);
  if (st != FG_OK) return st;
  const bool f8 = d->w_dtype == FG_E4M3;
  if (expert_offsets == nullptr) return fail(FG_ERR_INVALID_ARG, "%s: expert_offsets is NULL", fn);
  if (d->T > 0 && (tokens == nullptr || router_logits == nullptr || w_gateup == nullptr || w_down == nullptr ||
                   out == nullptr || topk_idx == nullptr || topk_w == nullptr || perm == nullptr))
    return fail(FG_ERR_INVALID_ARG, "%s: a required pointer is NULL", fn);
  if (f8 && (s_gateup == nullptr || s_down == nullptr))
    return fail(FG_ERR_INVALID_ARG, "%s: e4m3 weights need s_gateup and s_down", fn);
  const void* p16[] = {tokens, router_logits, w_gateup, w_down, out, topk_idx, topk_w, perm, expert_offsets,
                       s_gateup, s_down, workspace};
  for (const void* p : p16)
    if (!aligned16(p)) return fail(FG_ERR_ALIGNMENT, "%s: every pointer must be 16-byte aligned", fn);
  const MoeLayout L = layout(*d);
  if (workspace == nullptr || ws_bytes < L.total)
    return fail(FG_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, L.total,
                workspace ? ws_bytes : (size_t)0);

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  int32_t* tile_off = reinterpret_cast<int32_t*>(ws + L.tile_off);
  const int64_t S = L.S;
  const int T = (int)d->T;
  if (T == 0) {
    // no tokens: every expert is empty (a fill kernel, not a memset node, so
    // that the call may be captured into a graph)
    hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)((d->E + 1 + 255) / 256)), dim3(256), 0, s, expert_offsets,
                       d->E + 1, 0);
    return check_launch(fn);
  }
  const char* a_tokens = static_cast<const char*>(tokens);
  float* sx = reinterpret_cast<float*>(ws + L.sx);
  if (f8) {
    hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)((d->T + 3) / 4)), dim3(256), 0, s,
                       static_cast<const uint16_t*>(tokens), d->T, d->H, reinterpret_cast<uint8_t*>(ws + L.xq), sx);
    a_tokens = ws + L.xq;
  }
  hipLaunchKernelGGL(moe_route_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, router_logits, T, d->E,
                     d->top_k, topk_idx, topk_w);
  if (S <= PERM_LDS_SLOTS)
    hipLaunchKernelGGL(moe_permute_kernel<true>, dim3(1), dim3(PERM_THREADS), 0, s, topk_idx, (int)S, d->E, L.BM,
                       expert_offsets, tile_off, perm);
  else
    hipLaunchKernelGGL(moe_permute_kernel<false>, dim3(1), dim3(PERM_THREADS), 0, s, topk_idx, (int)S, d->E,
                       L.BM, expert_offsets, tile_off, perm);

  GroupedArgs g;
  g.perm = perm;
  g.offsets = expert_offsets;
  g.tile_off = tile_off;
  g.topk_w = topk_w;
  g.E = d->E;
  g.k = d->top_k;
  g.I = d->I;
  g.alpha = d->swiglu_alpha;
  g.limit = d->swiglu_limit;
  g.interleaved = d->gateup_interleaved;

  // gate/up: [S, H] × [2I, H]ᵀ → h [S, I]
  g.A = a_tokens;
  g.W = static_cast<const char*>(w_gateup);
  g.a_scale = f8 ? sx : nullptr;
  g.w_scale = s_gateup;
  g.out = ws + L.h;
  g.K = d->H;
  g.Nw = 2 * d->I;
  g.ldo = d->I;
  g.tiles_n = (int)(d->I / 64);
  if (f8) {
    if (L.BM == 128) launch_grouped<GF8Big, EPI_GATEUP>(g, S, s);
    else launch_grouped<GF8Small, EPI_GATEUP>(g, S, s);
  } else {
    if (L.BM == 128) launch_grouped<GBf16Big, EPI_GATEUP>(g, S, s);
    else launch_grouped<GBf16Small, EPI_GATEUP>(g, S, s);
  }

  // down: [S, I] × [H, I]ᵀ → y_slot [S, H] (× routing weight, scattered to slot order)
  const char* hA = ws + L.h;
  float* sh = reinterpret_cast<float*>(ws + L.sh);
  if (f8) {
    hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)((S + 3) / 4)), dim3(256), 0, s,
                       reinterpret_cast<const uint16_t*>(ws + L.h), S, d->I,
                       reinterpret_cast<uint8_t*>(ws + L.hq), sh);
    hA = ws + L.hq;
  }
  g.A = hA;
  g.W = static_cast<const char*>(w_down);
  g.a_scale = f8 ? sh : nullptr;
  g.w_scale = s_down;
  g.out = ws + L.y;
  g.K = d->I;
  g.Nw = d->H;
  g.ldo = d->H;
  g.tiles_n = (int)((d->H + 127) / 128);
  if (f8) {
    if (L.BM == 128) launch_grouped<GF8Big, EPI_DOWN>(g, S, s);
    else launch_grouped<GF8Small, EPI_DOWN>(g, S, s);
  } else {
    if (L.BM == 128) launch_grouped<GBf16Big, EPI_DOWN>(g, S, s);
    else launch_grouped<GBf16Small, EPI_DOWN>(g, S, s);
  }

  const int64_t threads = d->T * (d->H / 8);
  hipLaunchKernelGGL(moe_finalize_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const uint16_t*>(ws + L.y), static_cast<uint16_t*>(out), T, d->H,
                     d->top_k);
  return check_launch(fn);
}
