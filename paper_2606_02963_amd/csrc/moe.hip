// moe.hip — one MoE expert-FFN step of a gpt-oss-20b-like layer.
//
// Launch sequence on the caller's stream, with no host synchronisation (the
// per-expert counts never leave the device):
//   [e4m3 only] quantise tokens per row          quantize_rows_kernel
//   route: top-k + softmax per token, and the    moe_route_kernel
//     expert histogram of each block of tokens
//   offsets, stable permutation, m-tile prefix   moe_place_kernel
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
// route: a workgroup covers ROUTE_TOKENS tokens. Their logits are first
// staged in LDS with one coalesced pass; then one thread per token keeps the
// top-k in a list sorted by the key (value descending, index ascending), so
// ties go to the lower expert index, and takes the softmax over the k
// selected logits. The workgroup also forms the expert histogram of its
// slots (LDS atomics: integer counts do not depend on the order of the adds).
//
// place: the stable permutation. The slots of a workgroup's tokens are
// split into contiguous per-wave ranges; a slot's position is
//   offsets[e] + Σ_{b' < b} count[b'][e] + Σ_{w' < w} count_w'[e]
//   + (earlier slots of expert e in the wave's own range),
// i.e. its rank in the sort by (expert, slot id). Inside a wave, 64-slot
// chunks are processed in order and each distinct expert of a chunk takes
// one ballot. No atomics decide a position, so the result is unique and
// bit-reproducible. Workgroup 0 also writes offsets and the m-tile prefix
// the grouped GEMMs read. When one workgroup covers every token, route and
// place run in the same launch.

constexpr int ROUTE_TOKENS = 64;          // tokens per route / place workgroup
constexpr int ROUTE_WAVES = 4;
constexpr int PLACE_WAVES = 4;

__device__ __forceinline__ bool key_wins(float v, int i, float bv, int bi) {
  return (v > bv) | ((v == bv) & (i < bi));
}

// Stable placement of the slots [s_begin, s_begin + n_slots) by NW waves.
// off[e]: the global position of this workgroup's first slot of expert e.
// wrun: NW × EMAX ints of LDS. Ends after writing perm.
template <int NW>
__device__ __forceinline__ void place_slots(const int32_t* topk_idx, int s_begin, int n_slots, int E,
                                            const int* off, int (*wrun)[EMAX], int32_t* perm) {
  constexpr int CH = (KMAX * ROUTE_TOKENS / NW + 63) / 64;     // 64-slot chunks per wave, at most
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int e = threadIdx.x; e < E; e += 64 * NW)
#pragma unroll
    for (int w = 0; w < NW; ++w) wrun[w][e] = 0;
  __syncthreads();
  const int per_wave = (n_slots + NW - 1) / NW;
  const int s0 = s_begin + wave * per_wave;
  const int s_end = s_begin + n_slots;
  const unsigned long long lt = (1ull << lane) - 1ull;
  int my_e[CH], my_rank[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    my_e[c] = -1;
    my_rank[c] = 0;
    if (c * 64 >= per_wave) continue;        // uniform
    const int s = s0 + c * 64 + lane;
    const bool valid = (c * 64 + lane < per_wave) && s < s_end;
    const int e = valid ? topk_idx[s] : -1;
    my_e[c] = e;
    unsigned long long pending = __ballot(valid);
    while (pending) {
      const int leader = __ffsll((long long)pending) - 1;
      const int le = __shfl(e, leader, 64);
      const unsigned long long m = __ballot(valid && e == le);
      const int run = wrun[wave][le];
      if (valid && e == le) my_rank[c] = run + __popcll(m & lt);
      if (lane == leader) wrun[wave][le] = run + __popcll(m);
      pending &= ~m;
    }
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int e = my_e[c];
    if (e < 0) continue;
    int r = off[e] + my_rank[c];
    for (int w = 0; w < wave; ++w) r += wrun[w][e];
    perm[r] = s0 + c * 64 + lane;
  }
}

// Exclusive prefix of the per-expert totals `tot` (in place) by one thread;
// workgroup 0 also publishes offsets and the m-tile prefix.
__device__ __forceinline__ void publish_offsets(int* tot, int E, int BM, int32_t* offsets, int32_t* tile_off) {
  if (threadIdx.x == 0) {
    int acc = 0, tacc = 0;
    for (int e = 0; e < E; ++e) {
      const int c = tot[e];
      tot[e] = acc;
      if (blockIdx.x == 0) {
        offsets[e] = acc;
        tile_off[e] = tacc;
      }
      acc += c;
      tacc += (c + BM - 1) / BM;
    }
    if (blockIdx.x == 0) {
      offsets[E] = acc;
      tile_off[E] = tacc;
    }
  }
  __syncthreads();
}

template <bool FUSED_PLACE>
__global__ __launch_bounds__(64 * ROUTE_WAVES) void moe_route_kernel(const float* logits, int T, int E, int k,
                                                                     int32_t* topk_idx, float* topk_w,
                                                                     int32_t* block_counts, int BM,
                                                                     int32_t* offsets, int32_t* tile_off,
                                                                     int32_t* perm) {
  // row pitch E + 1 floats: thread t reading its row's logit e hits bank (t·(E+1) + e) mod 64
  __shared__ float lg[ROUTE_TOKENS * (EMAX + 1)];
  __shared__ int hist[EMAX];
  __shared__ int wrun[FUSED_PLACE ? ROUTE_WAVES : 1][EMAX];
  const int t0 = blockIdx.x * ROUTE_TOKENS;
  const int nt = T - t0 < ROUTE_TOKENS ? T - t0 : ROUTE_TOKENS;
  const int pitch = E + 1;
  for (int e = threadIdx.x; e < E; e += 64 * ROUTE_WAVES) hist[e] = 0;
  const float* src = logits + (int64_t)t0 * E;
  const int n = nt * E;
  constexpr int UNR = 8;                     // loads in flight per thread before the LDS stores
  for (int i0 = threadIdx.x; i0 < n; i0 += 64 * ROUTE_WAVES * UNR) {
    float x[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u * 64 * ROUTE_WAVES;
      x[u] = i < n ? src[i] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u * 64 * ROUTE_WAVES;
      if (i < n) lg[(i / E) * pitch + i % E] = x[u];
    }
  }
  __syncthreads();
  const int tt = threadIdx.x;
  if (tt < nt) {
    // insertion into a list sorted by (value descending, index ascending);
    // experts arrive in ascending order, an entry is displaced only by a
    // larger key, and the compare-exchange is branch-free
    float bv[KMAX];
    int bi[KMAX];
#pragma unroll
    for (int p = 0; p < KMAX; ++p) {
      bv[p] = -INFINITY;
      bi[p] = -1;
    }
    const float* row = lg + tt * pitch;
    for (int e = 0; e < E; ++e) {
      const float x = row[e];
      float v = x != x ? -INFINITY : x;     // a NaN logit ranks as −∞, so k experts are always selected
      int id = e;
#pragma unroll
      for (int p = 0; p < KMAX; ++p) {
        const bool take = (bi[p] < 0) | key_wins(v, id, bv[p], bi[p]);
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
    const int t = t0 + tt;
#pragma unroll
    for (int p = 0; p < KMAX; ++p) {
      if (p < k) {
        topk_idx[(int64_t)t * k + p] = bi[p];
        topk_w[(int64_t)t * k + p] = ex[p] / sum;
        atomicAdd(&hist[bi[p]], 1);
      }
    }
  }
  __syncthreads();
  if constexpr (FUSED_PLACE) {
    // the only workgroup: its histogram is the total; topk_idx written above
    // by this workgroup is visible after the barrier
    publish_offsets(hist, E, BM, offsets, tile_off);
    place_slots<ROUTE_WAVES>(topk_idx, 0, T * k, E, hist, wrun, perm);
  } else {
    for (int e = threadIdx.x; e < E; e += 64 * ROUTE_WAVES) block_counts[(int64_t)blockIdx.x * E + e] = hist[e];
  }
}

__global__ __launch_bounds__(64 * PLACE_WAVES) void moe_place_kernel(const int32_t* topk_idx, const int32_t* block_counts,
                                                                     int S, int E, int k, int nblocks, int BM,
                                                                     int32_t* offsets, int32_t* tile_off,
                                                                     int32_t* perm) {
  __shared__ int tot[EMAX];
  __shared__ int before[EMAX];
  __shared__ int wrun[PLACE_WAVES][EMAX];
  for (int e = threadIdx.x; e < E; e += 64 * PLACE_WAVES) {
    tot[e] = 0;
    before[e] = 0;
  }
  __syncthreads();
  // per-expert totals and the counts of earlier workgroups, summed by all
  // threads in parallel (integer LDS atomics: order-independent)
  const int n = nblocks * E;
  constexpr int UNR = 8;                     // loads in flight per thread before the LDS adds
  for (int i0 = threadIdx.x; i0 < n; i0 += 64 * PLACE_WAVES * UNR) {
    int c[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u * 64 * PLACE_WAVES;
      c[u] = i < n ? block_counts[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u * 64 * PLACE_WAVES;
      if (i < n) {
        atomicAdd(&tot[i % E], c[u]);
        if (i / E < (int)blockIdx.x) atomicAdd(&before[i % E], c[u]);
      }
    }
  }
  __syncthreads();
  publish_offsets(tot, E, BM, offsets, tile_off);
  for (int e = threadIdx.x; e < E; e += 64 * PLACE_WAVES) before[e] += tot[e];
  __syncthreads();
  const int s_begin = blockIdx.x * ROUTE_TOKENS * k;
  const int n_slots = (S - s_begin) < ROUTE_TOKENS * k ? S - s_begin : ROUTE_TOKENS * k;
  place_slots<PLACE_WAVES>(topk_idx, s_begin, n_slots, E, before, wrun, perm);
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
  int E, k;
  int tiles_n;             // n-tiles of the output
  int tiles_n_grid;        // n-tiles per grid row: tiles_n rounded up to a multiple of 8
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
  // n fastest; with tiles_n_grid a multiple of 8 and workgroups dealt to the
  // 8 XCDs round-robin, every m-tile of a given n-tile runs on the same XCD,
  // so the weight tile is fetched into one L2 and reused there
  const int tn = blockIdx.x % a.tiles_n_grid;
  const int mt = blockIdx.x / a.tiles_n_grid;
  if (tn >= a.tiles_n || mt >= a.tile_off[a.E]) return;
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

// Prefill tiles are 128 × 128 (4 waves): on the T = 4096 step they measured
// faster than 192- and 256-row tiles, whose ragged last m-tile per expert
// (n_e ≈ 512 ± 22 slots) wastes more of the matrix cores.
typedef Tile<In::BF16, 128, 128> GBf16Big;
typedef Tile<In::BF16, 32, 128> GBf16Small;
typedef Tile<In::E4M3, 128, 128> GF8Big;
typedef Tile<In::E4M3, 32, 128> GF8Small;

struct MoeLayout {
  int64_t S;
  int BM;
  int nblocks;             // route / place workgroups
  size_t tile_off, counts, h, y, xq, sx, hq, sh, total;
};

static size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

// Row tile of the grouped GEMMs: the big tile when experts average more than
// 48 slots, else the 32-row tile (decode: a handful of rows per expert, weight
// streaming). The launch dispatches on the same predicate, and the m-tile
// prefix is built with the chosen tile's BM.
static bool use_big_tiles(int64_t S, int E) { return S > (int64_t)48 * E; }
static int pick_bm(int64_t S, int E) { return use_big_tiles(S, E) ? GBf16Big::BM : GBf16Small::BM; }
static_assert(GBf16Big::BM == GF8Big::BM && GBf16Small::BM == GF8Small::BM,
              "bf16 and e4m3 tiles must share BM: one m-tile prefix serves both");

static MoeLayout layout(const moe_desc& d) {
  MoeLayout L;
  L.S = d.T * d.top_k;
  L.BM = pick_bm(L.S, d.E);
  size_t o = 0;
  L.nblocks = (int)((d.T + ROUTE_TOKENS - 1) / ROUTE_TOKENS);
  L.tile_off = o;
  o = align_up(o + sizeof(int32_t) * (size_t)(d.E + 1));
  L.counts = o;
  o = align_up(o + sizeof(int32_t) * (size_t)L.nblocks * (size_t)d.E);
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

// n-tiles: gate/up tiles cover BN/2 columns of h (BN weight rows, gate and
// up interleaved), down tiles BN columns of the output.
template <class TL, int EPI>
static void launch_grouped(GroupedArgs a, int64_t S, hipStream_t s) {
  a.tiles_n = EPI == EPI_GATEUP ? (int)(a.I / (TL::BN / 2)) : (int)((a.Nw + TL::BN - 1) / TL::BN);
  a.tiles_n_grid = (a.tiles_n + 7) / 8 * 8;
  const int64_t mtiles = (S + (int64_t)a.E * (TL::BM - 1)) / TL::BM;
  const unsigned grid = (unsigned)(mtiles * a.tiles_n_grid);
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
  int32_t* counts = reinterpret_cast<int32_t*>(ws + L.counts);
  if (L.nblocks == 1) {
    hipLaunchKernelGGL(moe_route_kernel<true>, dim3(1), dim3(64 * ROUTE_WAVES), 0, s, router_logits, T, d->E,
                       d->top_k, topk_idx, topk_w, counts, L.BM, expert_offsets, tile_off, perm);
  } else {
    hipLaunchKernelGGL(moe_route_kernel<false>, dim3((unsigned)L.nblocks), dim3(64 * ROUTE_WAVES), 0, s,
                       router_logits, T, d->E, d->top_k, topk_idx, topk_w, counts, L.BM, expert_offsets, tile_off,
                       perm);
    hipLaunchKernelGGL(moe_place_kernel, dim3((unsigned)L.nblocks), dim3(64 * PLACE_WAVES), 0, s, topk_idx, counts,
                       (int)S, d->E, d->top_k, L.nblocks, L.BM, expert_offsets, tile_off, perm);
  }

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
  if (f8) {
    if (use_big_tiles(S, d->E)) launch_grouped<GF8Big, EPI_GATEUP>(g, S, s);
    else launch_grouped<GF8Small, EPI_GATEUP>(g, S, s);
  } else {
    if (use_big_tiles(S, d->E)) launch_grouped<GBf16Big, EPI_GATEUP>(g, S, s);
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
  if (f8) {
    if (use_big_tiles(S, d->E)) launch_grouped<GF8Big, EPI_DOWN>(g, S, s);
    else launch_grouped<GF8Small, EPI_DOWN>(g, S, s);
  } else {
    if (use_big_tiles(S, d->E)) launch_grouped<GBf16Big, EPI_DOWN>(g, S, s);
    else launch_grouped<GBf16Small, EPI_DOWN>(g, S, s);
  }

  const int64_t threads = d->T * (d->H / 8);
  hipLaunchKernelGGL(moe_finalize_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const uint16_t*>(ws + L.y), static_cast<uint16_t*>(out), T, d->H,
                     d->top_k);
  return check_launch(fn);
}
