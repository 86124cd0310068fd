// moe.hip — one MoE expert-FFN step of a gpt-oss-20b-like layer.
//
// Launch sequence on the caller's stream, with no host synchronisation (the
// per-expert counts never leave the device):
//   route: top-k + softmax per token, and the    moe_route_kernel
//     expert histogram of each block of tokens;
//     [e4m3 only] the tokens quantised per row
//     by further blocks of the same launch
//   offsets, stable permutation, m-tile prefix   moe_place_kernel
//     (with one routing block: inside the routing launch)
//   grouped gate/up GEMM + clamped SwiGLU        grouped_kernel<.., EPI_GATEUP>
//   [e4m3 only] quantise h per row               quantize_rows_kernel
//   grouped down GEMM, fp32 slot outputs          grouped_kernel<.., EPI_DOWN>
//   finalize: Σ_j w_j·y over the k slots of a     moe_finalize_kernel
//     token, one rounding to bf16
// The token gather is folded into the gate/up GEMM's A-row addresses, and
// the scatter back to slot order into the down GEMM's store addresses, so no
// permuted copy of the tokens or of the outputs is ever materialised.
//
// Paper §IV-A optimises this block's decode kernels (MoE finalize, Table I);
// §V names optimising the whole MoE-MLP block jointly as the next step.
#include <hip/hip_runtime.h>
#include <math.h>

#include <atomic>
#include <type_traits>

#include "fg_host.hpp"
#include "fg_moe.hpp"
#include "fg_quant.hpp"
#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

__global__ void quantize_rows_kernel(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, float* s);

constexpr int KMAX = 8;       // largest supported top_k
constexpr int EMAX = 256;     // largest supported expert count

// ---------------------------------------------------------------------------
// route: a workgroup covers ROUTE_TOKENS tokens. Their logits are first
// staged in LDS with one coalesced pass; then four lanes per token select the
// top-k by descending key (value descending, ties to the lower expert index)
// and take the softmax over the k selected logits. The workgroup also forms
// the expert histogram of its slots (LDS atomics: integer counts do not
// depend on the order of the adds).
//
// place: the stable permutation. A slot's position is
//   offsets[e] + Σ_{b' < b} count[b'][e] + (earlier slots of expert e in
//   its own workgroup's range),
// i.e. its rank in the sort by (expert, slot id); the last term comes from
// per-expert slot bitmasks. No atomic decides a position, so the result is
// unique and bit-reproducible. Workgroup 0 also writes offsets and the
// m-tile prefix the grouped GEMMs read. When one workgroup covers every
// token, route and place run in the same launch.

constexpr int ROUTE_TOKENS = 64;          // tokens per route / place workgroup
constexpr int ROUTE_WAVES = 4;            // four lanes per token
static_assert(ROUTE_WAVES * 64 == 4 * ROUTE_TOKENS, "route workgroups hold four lanes per token");
constexpr int PLACE_WAVES = 4;

// Sortable 64-bit key of (logit, expert). The float's bits are mapped so that
// unsigned order is numeric order (negative values: all bits flipped;
// non-negative: sign bit set). −0 is first made +0 so that the two zeros,
// which compare equal, tie-break by index like any equal pair. A NaN logit
// ranks as −∞.
__device__ __forceinline__ uint64_t logit_key(float v, int e) {
  v = v != v ? -INFINITY : (v == 0.0f ? 0.0f : v);
  const uint32_t b = __float_as_uint(v);
  const uint32_t o = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)o << 32) | (uint32_t)(EMAX - 1 - e);
}
__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t o = (uint32_t)(key >> 32);
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// Stable placement of the slots [s_begin, s_begin + n_slots) of one
// workgroup (n_slots ≤ PLACE_MAX_SLOTS). Each slot sets its bit in its
// expert's slot mask (LDS atomicOr: the result does not depend on the
// order); a slot's rank among its expert's slots is then the popcount of
// the mask below its own bit, so the position off[e] + rank is its place in
// the sort by (expert, slot id). off[e]: the global position of this
// workgroup's first slot of expert e. masks: E × PLACE_WORDS words of LDS.
constexpr int PLACE_MAX_SLOTS = KMAX * ROUTE_TOKENS;
constexpr int PLACE_WORDS = PLACE_MAX_SLOTS / 32;

template <int NT>
__device__ __forceinline__ void place_slots(const int32_t* topk_idx, int s_begin, int n_slots, int E,
                                            const int* off, uint32_t* masks, int32_t* perm) {
  constexpr int PER = PLACE_MAX_SLOTS / NT;
  for (int i = threadIdx.x; i < E * PLACE_WORDS; i += NT) masks[i] = 0u;
  __syncthreads();
  int my_e[PER];
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    const int sl = threadIdx.x + c * NT;
    my_e[c] = sl < n_slots ? topk_idx[s_begin + sl] : -1;
    if (my_e[c] >= 0) atomicOr(&masks[my_e[c] * PLACE_WORDS + (sl >> 5)], 1u << (sl & 31));
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    const int e = my_e[c];
    if (e < 0) continue;
    const int sl = threadIdx.x + c * NT;
    const uint32_t* m = masks + e * PLACE_WORDS;
    int rank = __popc(m[sl >> 5] & ((1u << (sl & 31)) - 1u));
    for (int w = 0; w < (sl >> 5); ++w) rank += __popc(m[w]);
    perm[off[e] + rank] = s_begin + sl;
  }
}

// Exclusive prefix of the per-expert totals `tot` (in place) and of their
// m-tile counts, by wave 0: lane l owns experts 4l .. 4l + 3 (E ≤ 256), then a
// scan of the lane sums over the ceil(E/4) lanes that hold experts.
// Workgroup 0 also publishes offsets and the m-tile prefix. BM is a power of
// two.
__device__ __forceinline__ void publish_offsets(int* tot, int E, int BM, int32_t* offsets, int32_t* tile_off) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int bm_shift = __builtin_ctz((unsigned)BM);
    const int nlanes = (E + 3) >> 2;
    int c[4], tc[4], s = 0, ts = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < E ? tot[e] : 0;
      tc[q] = (c[q] + BM - 1) >> bm_shift;
      s += c[q];
      ts += tc[q];
    }
    int incl = s, tincl = ts;
    for (int d = 1; d < nlanes; d <<= 1) {
      const int y = __shfl_up(incl, d, 64), ty = __shfl_up(tincl, d, 64);
      if (lane >= d) {
        incl += y;
        tincl += ty;
      }
    }
    int acc = incl - s, tacc = tincl - ts;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      if (e < E) {
        tot[e] = acc;
        if (blockIdx.x == 0) {
          offsets[e] = acc;
          tile_off[e] = tacc;
        }
      }
      acc += c[q];
      tacc += tc[q];
    }
    if (blockIdx.x == 0 && lane == nlanes - 1) {
      offsets[E] = incl;
      tile_off[E] = tincl;
    }
  }
  __syncthreads();
}

// Largest of a 64-bit key over the 4 lanes of a quad (DPP quad permutes
// lane ^ 1 and lane ^ 2 on both halves).
__device__ __forceinline__ uint64_t quad_max_u64(uint64_t m) {
  uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
  uint64_t o;
  lo = (uint32_t)m;
  o = ((uint64_t)(uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, 0xB1, 0xF, 0xF, false) << 32) |
      (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, 0xB1, 0xF, 0xF, false);
  m = o > m ? o : m;
  lo = (uint32_t)m;
  hi = (uint32_t)(m >> 32);
  o = ((uint64_t)(uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, 0x4E, 0xF, 0xF, false) << 32) |
      (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, 0x4E, 0xF, 0xF, false);
  return o > m ? o : m;
}
__device__ __forceinline__ float quad_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  return v;
}

template <bool FUSED_PLACE>
__global__ __launch_bounds__(64 * ROUTE_WAVES) void moe_route_kernel(const float* logits, int T, int E, int k,
                                                                     int32_t* topk_idx, float* topk_w,
                                                                     int32_t* block_counts, int BM,
                                                                     int32_t* offsets, int32_t* tile_off,
                                                                     int32_t* perm, const uint16_t* xq_src,
                                                                     int64_t H, uint8_t* xq, float* sx) {
  // Routing shares its launch with the e4m3 quantisation of the tokens
  // (independent work): the blocks after the routing blocks take four token
  // rows each.
  const int rblocks = (T + ROUTE_TOKENS - 1) / ROUTE_TOKENS;
  if ((int)blockIdx.x >= rblocks) {
    quantize_row_wave(xq_src, T, H, xq, sx, (int64_t)(blockIdx.x - rblocks) * 4 + (threadIdx.x >> 6));
    return;
  }
  // row pitch E + 1 floats: thread t reading its row's logit e hits bank (t·(E+1) + e) mod 64
  __shared__ float lg[ROUTE_TOKENS * (EMAX + 1)];
  __shared__ int hist[EMAX];
  __shared__ int32_t chosen[FUSED_PLACE ? ROUTE_TOKENS * KMAX : 1];   // the block's slots, for placement
  __shared__ uint32_t masks[FUSED_PLACE ? EMAX * PLACE_WORDS : 1];
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
  // four lanes per token: lane `sub` scans experts sub, sub + 4, ...; each
  // pass takes the largest key below the previous winner, as a max over the
  // lane's keys followed by a max over the quad
  const int tt = threadIdx.x >> 2, sub = threadIdx.x & 3;
  const bool active = tt < nt;
  const float* row = lg + (active ? tt : 0) * pitch;
  uint64_t win = ~0ull;
  int sel_i = -1;           // lane q of the quad keeps selection q (and q + 4)
  int sel_i2 = -1;
  float sel_v = -INFINITY, sel_v2 = -INFINITY, top = -INFINITY;
  // E ≤ 32: the lane's (at most 8) keys stay in registers for all k passes
  constexpr int KPL = 8;
  uint64_t keys[KPL];
  const bool in_regs = E <= 4 * KPL;
  if (in_regs) {
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
      const int e = sub + 4 * u;
      keys[u] = e < E ? logit_key(row[e], e) : 0ull;
    }
  }
  for (int j = 0; j < k; ++j) {
    uint64_t m = 0;
    if (in_regs) {
#pragma unroll
      for (int u = 0; u < KPL; ++u) m = (keys[u] < win && keys[u] > m) ? keys[u] : m;
    } else {
      uint64_t part[4] = {0, 0, 0, 0};
      for (int e0 = sub; e0 < E; e0 += 16) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + 4 * u;
          if (e < E) {
            const uint64_t key = logit_key(row[e], e);
            part[u] = (key < win && key > part[u]) ? key : part[u];
          }
        }
      }
      m = part[0] > part[1] ? part[0] : part[1];
      const uint64_t m2 = part[2] > part[3] ? part[2] : part[3];
      m = m > m2 ? m : m2;
    }
    win = quad_max_u64(m);
    const int e = EMAX - 1 - (int)(win & 0xffffffffu);
    const float v = key_value(win);
    if (j == 0) top = v;
    if (j == sub) {
      sel_i = e;
      sel_v = v;
    }
    if (j == sub + 4) {
      sel_i2 = e;
      sel_v2 = v;
    }
  }
  const float ex = sub < k ? expf(sel_v - top) : 0.0f;
  const float ex2 = sub + 4 < k ? expf(sel_v2 - top) : 0.0f;
  const float sum = quad_sum(ex + ex2);
  if (active) {
    const int t = t0 + tt;
    if (sub < k) {
      topk_idx[(int64_t)t * k + sub] = sel_i;
      topk_w[(int64_t)t * k + sub] = ex / sum;
      atomicAdd(&hist[sel_i], 1);
      if constexpr (FUSED_PLACE) chosen[tt * k + sub] = sel_i;
    }
    if (sub + 4 < k) {
      topk_idx[(int64_t)t * k + sub + 4] = sel_i2;
      topk_w[(int64_t)t * k + sub + 4] = ex2 / sum;
      atomicAdd(&hist[sel_i2], 1);
      if constexpr (FUSED_PLACE) chosen[tt * k + sub + 4] = sel_i2;
    }
  }
  __syncthreads();
  if constexpr (FUSED_PLACE) {
    // the only workgroup: its histogram is the total, and its slots' experts
    // are in LDS (no round trip through the topk_idx stores)
    publish_offsets(hist, E, BM, offsets, tile_off);
    place_slots<64 * ROUTE_WAVES>(chosen, 0, T * k, E, hist, masks, perm);
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
  __shared__ uint32_t masks[EMAX * PLACE_WORDS];
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
  place_slots<64 * PLACE_WAVES>(topk_idx, s_begin, n_slots, E, before, masks, perm);
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
  char* out;               // gate/up: h [S, I] bf16 (expert order); down: y_slot [S, H] fp32 (slot order)
  int E, k;
  int tiles_n;             // n-tiles of the output
  int tiles_n_grid;        // n-tiles per grid row: tiles_n rounded up to a multiple of 8
  int64_t K;               // contraction length in elements
  int64_t Nw;              // weight rows per expert: 2I or H
  int64_t I;               // intermediate size (gate/up pairing)
  int64_t ldo;             // output row length in elements
  float alpha, limit;
  int interleaved;
  uint32_t a_bytes;        // gate/up: bytes of the token matrix when at most 2^31
};

// Gathered rows of a matrix of at most 2^31 bytes: one buffer descriptor
// over the whole matrix and a 32-bit byte offset per owned row, so the
// stage loads are MUBUF loads with the LDS bit, like the strided rows (BufRows).
// (With the global-segment form of the direct load in the loop, the
// compiler waited for every LDS fragment read of a stage before its first
// MFMA; with MUBUF loads it waits for each MFMA's own operands.) Rows past
// the matrix edge take the offset of any valid row, as in RowSet.
template <int NLD>
struct GatherRows {
  i32x4 rsrc;          // wave-uniform
  uint32_t row[NLD];   // byte offset of each owned row
  uint32_t cst;        // byte offset of the fetched chunk (see above)

  // `base` and `bytes` (≤ 2^31) must be uniform across the wave.
  __device__ __forceinline__ void init(const char* base, uint32_t bytes) {
    const i32x4 r = make_buffer_rsrc(base, bytes);
    rsrc = i32x4{__builtin_amdgcn_readfirstlane(r[0]), __builtin_amdgcn_readfirstlane(r[1]),
                 __builtin_amdgcn_readfirstlane(r[2]), __builtin_amdgcn_readfirstlane(r[3])};
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    cst = static_cast<uint32_t>(((lane & 7) ^ (lane >> 3) ^ (wave & 1)) * 16);
  }

  template <int NWAVES>
  __device__ __forceinline__ void stage(int64_t kbyte, char* sbase) const {
    static_assert(NWAVES % 2 == 0, "the fetched chunk assumes an even wave count");
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int p = 0; p < NLD; ++p) {
      char* dst = sbase + (wave + NWAVES * p) * 1024;
      fg_raw_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(dst), 16,
                             row[p] + cst + static_cast<uint32_t>(kbyte), 0, 0, 0);
    }
  }

  // Every load is issued before the first LDS write (one memory round trip);
  // chunks past kbytes get an out-of-range offset and read as zero.
  template <int RS>
  __device__ __forceinline__ void tail(int64_t kbyte, int64_t kbytes, char* sbase) const {
    const int c = threadIdx.x & 7;
    const int r0 = threadIdx.x >> 3;
    const int64_t off = kbyte + c * 16;
    const bool in = off < kbytes;
    i32x4 v[NLD];
#pragma unroll
    for (int p = 0; p < NLD; ++p)
      v[p] = fg_raw_buffer_load_b128(rsrc, in ? row[p] + static_cast<uint32_t>(off) : 0x80000000u, 0, 0);
#pragma unroll
    for (int p = 0; p < NLD; ++p) *reinterpret_cast<i32x4*>(sbase + lds_off(r0 + RS * p, c)) = v[p];
  }
};

// LDS of a grouped workgroup: the main loop's two stages, or the bf16 h
// staging of the gate/up epilogue.
template <class TL>
struct GroupedLds {
  static constexpr int OUT_STAGE = TL::BM * (TL::BN * 2 + 16);
  static constexpr int BYTES = TL::LOOP_LDS > OUT_STAGE ? TL::LOOP_LDS : OUT_STAGE;
};

// Weight row of tile-local B row ρ. Gate/up tiles interleave 16-row blocks:
// block f (ρ/16) is gate (f even) or up (f odd) of output columns
// (f/2)·16 .. +15, so a lane's accumulators for fragment pairs (2q, 2q+1)
// hold matching gate and up values.
// Columns of h past I (the ragged last n-tile) read the last column's rows;
// their results are never stored.
template <class TL, int EPI>
__device__ __forceinline__ int64_t weight_row(const GroupedArgs& a, int tn, int rho) {
  if constexpr (EPI == EPI_GATEUP) {
    const int f = rho >> 4;
    int64_t hc = (int64_t)tn * (TL::BN / 2) + (f >> 1) * 16 + (rho & 15);
    hc = hc < a.I ? hc : a.I - 1;
    const int up = f & 1;
    return a.interleaved ? 2 * hc + up : up * a.I + hc;
  } else {
    const int64_t n = (int64_t)tn * TL::BN + rho;
    return n < a.Nw ? n : a.Nw - 1;
  }
}

// WIDE: the gate/up token matrix exceeds 2^31 bytes, so its gathered rows
// are addressed by 64-bit pointers (RowSet) instead of 32-bit offsets into
// one buffer descriptor (GatherRows).
template <class TL, int EPI, bool WIDE>
__global__ __launch_bounds__(TL::THREADS) __attribute__((amdgpu_waves_per_eu(2))) void grouped_kernel(GroupedArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[GroupedLds<TL>::BYTES];
  // The m-tile prefix and the expert offsets, read once per workgroup into
  // registers (entry i in lane i mod 64, register i / 64; E ≤ 256): the
  // expert of an m-tile is then the number of experts whose tiles end at or
  // before it (a ballot), and its offsets come from lane shuffles, instead
  // of a chain of dependent global loads per tile.
  const int lane = threadIdx.x & 63;
  int toff_end[4], off_beg[4];   // tile_off[i + 1] (INT_MAX past E), offsets[i] (i < E)
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = lane + 64 * q;
    toff_end[q] = i < a.E ? a.tile_off[i + 1] : 0x7fffffff;
    off_beg[q] = i < a.E ? a.offsets[i] : 0;
  }
  // offsets[E], the end of the last expert's slots (entry 256 when E = 256
  // would fall past the four registers)
  const int off_end = a.offsets[a.E];
  auto pick = [&](const int (&v)[4], int i) {   // v[i / 64] of lane i mod 64 (i wave-uniform)
    const int q = i >> 6;
    const int x = q == 0 ? v[0] : q == 1 ? v[1] : q == 2 ? v[2] : v[3];
    return __shfl(x, i & 63, 64);
  };
  // Two tile orders. Both read the tile count from the device-side m-tile
  // prefix, and every workgroup reaches the end of its loop.
  //  * large (prefill) tiles: the real tiles, in expert-major order
  //    (expert, n-tile, m-tile), are cut into 8 contiguous ranges, and range
  //    x goes to the workgroups b ≡ x (mod 8), which the dispatcher places
  //    on XCD x, in order: entry (b >> 3) + t·(G / 8) in round t (one round
  //    when the grid covers every entry). An expert's weights are then streamed by
  //    one XCD (two at a range boundary) rather than by all eight, and the
  //    workgroups an XCD holds at a time cover every m-tile of the current
  //    expert over a run of n-tiles: each weight tile is used by all the
  //    expert's m-tiles while it is in that XCD's L2, and the expert's token
  //    rows stay there across the n-tiles.
  //  * small (decode) tiles, persistent (workgroup b takes tiles b, b + G, b + 2G, ... with
  //    G = gridDim.x a multiple of 8): tile t is (m-tile t / tiles_n_grid,
  //    n-tile t % tiles_n_grid), n fastest; with tiles_n_grid and G multiples
  //    of 8, every m-tile of a given n-tile runs on the same XCD, so the
  //    weight tile is fetched into one L2 and reused there.
  constexpr bool XCD_SPLIT = TL::BM > 32;
  const int mtiles = pick(toff_end, a.E - 1);
  const int ntiles = XCD_SPLIT ? 0x7fffffff : mtiles * a.tiles_n_grid;
  for (int t = XCD_SPLIT ? 0 : blockIdx.x; t < ntiles; t += XCD_SPLIT ? 1 : gridDim.x) {
  int e = 0, mt, tn;
  if constexpr (XCD_SPLIT) {
    // round t: workgroup b takes entry (b >> 3) + t·(G / 8) of range b mod 8
    const int total = mtiles * a.tiles_n;
    const int per = (total + 7) >> 3;
    const int l = (blockIdx.x >> 3) + t * (gridDim.x >> 3);
    const int u = (blockIdx.x & 7) * per + l;
    if (l >= per || u >= total) break;
#pragma unroll
    for (int q = 0; q < 4; ++q) e += __popcll(__ballot((int64_t)toff_end[q] * a.tiles_n <= u));
    const int first = e == 0 ? 0 : pick(toff_end, e - 1);
    const int me = pick(toff_end, e) - first;
    const int local = u - first * a.tiles_n;
    tn = local / me;
    mt = first + local % me;
  } else {
    tn = t % a.tiles_n_grid;
    mt = t / a.tiles_n_grid;
    if (tn >= a.tiles_n) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) e += __popcll(__ballot(toff_end[q] <= mt));
  }
  const int seg0 = pick(off_beg, e), seg1 = e + 1 < a.E ? pick(off_beg, e + 1) : off_end;
  const int r0 = seg0 + (mt - (e == 0 ? 0 : pick(toff_end, e - 1))) * TL::BM;
  const int64_t rowbytes = a.K * TL::ESIZE;
  const int tr = threadIdx.x >> 3;

  // A rows: gate/up gathers token rows through the permutation (a pointer
  // per row); down reads the expert's consecutive h rows. B rows: the
  // expert's weight rows, through one buffer descriptor and one offset per
  // lane (rows past the valid range read as zero; their columns are never
  // stored).
  using GRows = typename std::conditional<WIDE, RowSet<TL::A_LD>, GatherRows<TL::A_LD>>::type;
  using ARows = typename std::conditional<EPI == EPI_GATEUP, GRows, BufRows<TL::A_LD, TL::RSTRIDE>>::type;
  ARows ra;
  if constexpr (EPI == EPI_GATEUP) {
    if constexpr (!WIDE) ra.init(a.A, a.a_bytes);
#pragma unroll
    for (int p = 0; p < TL::A_LD; ++p) {
      int r = r0 + tr + TL::RSTRIDE * p;
      r = r < seg1 ? r : seg0;
      const int64_t tok = a.perm[r] / a.k;
      if constexpr (WIDE)
        ra.ptr[p] = a.A + tok * rowbytes;
      else
        ra.row[p] = static_cast<uint32_t>(tok * rowbytes);
    }
  } else {
    ra.init(a.A + (int64_t)r0 * rowbytes, seg1 - r0, TL::BM, rowbytes);
  }
  BufRows<TL::B_LD, TL::RSTRIDE> rb;
  const char* We = a.W + (int64_t)e * a.Nw * rowbytes;
  if constexpr (EPI == EPI_GATEUP) {
    // Thread t loads tile rows ρ = tr + RSTRIDE·p, which interleave 16-row
    // blocks of gate and up rows (weight_row): ρ is an up row when bit 4 of
    // ρ is set, and h column (ρ >> 5)·16 + (ρ & 15) of the tile. RSTRIDE is
    // a multiple of 32, so all rows of a thread are gate rows or all are up
    // rows (those of one wave alike: tr >> 4 = wave >> 1), RSTRIDE / 2 h
    // columns apart.
    static_assert(TL::RSTRIDE % 32 == 0 && TL::BN / 2 == (TL::RSTRIDE / 2) * TL::B_LD,
                  "gate/up B rows: RSTRIDE / 2 h columns per load");
    const int up = (tr >> 4) & 1;
    const int64_t col = (tr >> 5) * 16 + (tr & 15);
    const int64_t c0 = (int64_t)tn * (TL::BN / 2);
    const int64_t cols = a.I - c0 < TL::BN / 2 ? a.I - c0 : TL::BN / 2;    // valid h columns
    const int64_t step = a.interleaved ? 2 : 1;                              // rows per h column
    const char* base = We + (a.interleaved ? 2 * c0 + up : up * a.I + c0) * rowbytes;
    const uint32_t bytes = static_cast<uint32_t>(((cols - 1) * step + 1) * rowbytes);
    rb.init_rows(base, bytes, static_cast<uint32_t>(step * col * rowbytes),
                 static_cast<uint32_t>(step * (TL::RSTRIDE / 2) * rowbytes));
  } else {
    rb.init(We + (int64_t)tn * TL::BN * rowbytes, a.Nw - (int64_t)tn * TL::BN, TL::BN, rowbytes);
  }

  // e4m3 dequantisation factors (per accumulator row the scale of its
  // activation row, per column the weight-row scale), loaded before the K
  // loop so that their dependent loads (slot → token → scale) complete
  // behind it. The routing weight is applied in the finalize.
  float rs[TL::IN == In::E4M3 ? TL::FM : 1][4];
  float ws[TL::IN == In::E4M3 ? TL::FN : 1];
  if constexpr (TL::IN == In::E4M3) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int r = r0 + acc_row<TL>(fm, i);
        r = r < seg1 ? r : seg0;
        rs[fm][i] = EPI == EPI_GATEUP ? a.a_scale[a.perm[r] / a.k] : a.a_scale[r];
      }
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
      ws[fn] = a.w_scale[(int64_t)e * a.Nw + weight_row<TL, EPI>(a, tn, acc_col<TL>(fn))];
  }

  f32x4 acc[TL::FM][TL::FN];
  gemm_mainloop<TL>(ra, rb, rowbytes, lds, acc, seg1 - r0);

  const int l = threadIdx.x & 63, wave = threadIdx.x >> 6, wn = wave % TL::WN;
  if constexpr (TL::IN == In::E4M3) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[fm][fn][i] *= rs[fm][i] * ws[fn];
  }

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
          v = (u + 1.0f) * (g * fast_sigmoid(alpha * g));
          c = ((wn * TL::FN + fn) >> 1) * 16 + (l & 15);
          return true;
        },
        [&](int r) -> char* {
          const int row = r0 + r;
          return row < seg1 ? out + ((int64_t)row * ldo + c0) * 2 : nullptr;
        },
        (int)(a.I - c0 < TL::BN / 2 ? a.I - c0 : TL::BN / 2));
  } else {
    char* out = a.out;
    const int64_t ldo = a.ldo;
    const int n0 = tn * TL::BN;
    const int ncols = (int)(a.Nw - n0 < TL::BN ? a.Nw - n0 : TL::BN);
    // The slot outputs stay fp32; the finalize weights and sums them and
    // rounds once. They are stored straight from the
    // accumulators: for each accumulator row, 16 lanes write 64 contiguous
    // bytes, and the neighbouring fragments of the same row complete the
    // line in L2 (measured faster than staging the fp32 tile through LDS in
    // two column slabs: 350 vs 371 µs bf16, 261 vs 287 µs e4m3 on the
    // T = 4096 step). The slot id of each tile row goes through LDS once.
    int* slot_of = reinterpret_cast<int*>(lds);
    __syncthreads();
    for (int r = threadIdx.x; r < TL::BM; r += TL::THREADS) slot_of[r] = r0 + r < seg1 ? a.perm[r0 + r] : -1;
    __syncthreads();
    float* outf = reinterpret_cast<float*>(out);
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int slot = slot_of[acc_row<TL>(fm, i)];
        if (slot < 0) continue;
        float* dst = outf + (int64_t)slot * ldo + n0;
#pragma unroll
        for (int fn = 0; fn < TL::FN; ++fn) {
          const int c = acc_col<TL>(fn);
          if (c < ncols) dst[c] = acc[fm][fn][i];
        }
      }
  }
  // the next tile's loads overwrite the LDS this tile's store just read
  __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// finalize: out[t, :] = Σ_j w_j·y_slot[t·k + j, :], j ascending, fp32 sum,
// bf16 out (paper §IV-A, the MoE finalize kernel of Table I). One thread per
// 8 consecutive columns of a token; its K slot loads are all issued before
// the first add, so a launch costs one memory round trip whatever K is. The
// slot rows are bf16 and already weighted (the standalone Table I kernel,
// w_j = 1) or fp32 (inside the MoE step, where the down GEMM leaves them
// unrounded and unweighted, and w_j is the slot's routing weight).

template <int K, class Y>
__global__ __launch_bounds__(256) void moe_finalize_kernel(const Y* y_slot, const float* slot_w, uint16_t* out,
                                                           int T, int64_t H) {
  const int64_t cpt = H / 8;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = idx / cpt, c = idx % cpt;
  if (t >= T) return;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if constexpr (sizeof(Y) == 2) {
    i32x4 v[K];
#pragma unroll
    for (int j = 0; j < K; ++j) v[j] = *reinterpret_cast<const i32x4*>(y_slot + ((t * K + j) * H + c * 8));
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += bf16_bits_to_f32((uint16_t)(v[j][q] & 0xffff));
        acc[2 * q + 1] += bf16_bits_to_f32((uint16_t)((uint32_t)v[j][q] >> 16));
      }
  } else {
    f32x4 v[K][2];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        v[j][h] = *reinterpret_cast<const f32x4*>(y_slot + ((t * K + j) * H + c * 8 + h * 4));
    // the routing weights of the token's slots, when given
    float wj[K];
#pragma unroll
    for (int j = 0; j < K; ++j) wj[j] = slot_w != nullptr ? slot_w[t * K + j] : 1.0f;
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] += wj[j] * v[j][q >> 2][q & 3];
  }
  i32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = (int)((uint32_t)f32_to_bf16_bits(acc[2 * q]) | ((uint32_t)f32_to_bf16_bits(acc[2 * q + 1]) << 16));
  *reinterpret_cast<i32x4*>(out + (t * H + c * 8)) = o;
}

// Enqueue the finalize for top_k = k (1 .. KMAX) over slot rows of type Y,
// weighting slot p by w[p] when w is given (fp32 slot rows only).
template <class Y>
static hipError_t launch_finalize(const Y* y, const float* w, void* out, int64_t T, int64_t H, int k,
                                  hipStream_t s) {
  const int64_t threads = T * (H / 8);
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  uint16_t* o = static_cast<uint16_t*>(out);
  const int t = (int)T;
  switch (k) {
    case 1: return launch(moe_finalize_kernel<1, Y>, grid, block, 0, s, y, w, o, t, H);
    case 2: return launch(moe_finalize_kernel<2, Y>, grid, block, 0, s, y, w, o, t, H);
    case 3: return launch(moe_finalize_kernel<3, Y>, grid, block, 0, s, y, w, o, t, H);
    case 4: return launch(moe_finalize_kernel<4, Y>, grid, block, 0, s, y, w, o, t, H);
    case 5: return launch(moe_finalize_kernel<5, Y>, grid, block, 0, s, y, w, o, t, H);
    case 6: return launch(moe_finalize_kernel<6, Y>, grid, block, 0, s, y, w, o, t, H);
    case 7: return launch(moe_finalize_kernel<7, Y>, grid, block, 0, s, y, w, o, t, H);
    default: return launch(moe_finalize_kernel<8, Y>, grid, block, 0, s, y, w, o, t, H);
  }
}
static_assert(KMAX == 8, "launch_finalize instantiates top_k 1 .. 8");

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---------------------------------------------------------------------------
// host side

// Prefill tiles are 128 × 192 (4 waves, two workgroups per compute unit:
// 2 × 80 KB of LDS rings fill the 160 KB). 192 weight rows per stage cut the
// L2 → LDS bytes per FLOP by 17 % against 128 × 128 (13.0 vs 15.6 KB per
// MFLOP, 52 vs 62.5 B/clk per compute unit at the full MFMA rate); 192- and
// 256-row tiles lose more to the ragged last m-tile per
// expert (n_e ≈ 512 ± 22 slots), and 128 × 256 fits one workgroup per unit.
// Measured on the T = 4096 step: bf16 980–983 µs vs 1088–1090 µs with
// 128 × 128, e4m3 697 vs 710–713 µs; with the present kernels 256 × 256
// (8 waves, one workgroup per unit, waves of empty row halves idle) and
// 256 × 192 tiles take 1012 and 1052 µs against 939 µs. The bf16 prefill
// tile raises the wave priority over its MFMA clusters (927 vs 944 µs);
// the dense tiles do not (the LSE shape lost 3 % with it).
// Decode e4m3 tiles are 192 weight rows wide: a tile then streams
// 192 × H bytes, closer to the bf16 tile's 128 × 2H, so the per-tile start-up
// is amortised over more bytes, and 192 divides the gpt-oss geometry exactly
// (2880 = 30 × 96 h columns, 15 × 192 down rows). Measured: 161.8–162.2 µs vs
// 165.1 µs for 128-row tiles and 177 µs for 256 on the T = 64 step.
typedef Tile<In::BF16, 128, 192, 2, 2, true> GBf16Big;
typedef Tile<In::BF16, 32, 128> GBf16Small;
typedef Tile<In::E4M3, 128, 192> GF8Big;
typedef Tile<In::E4M3, 32, 192> GF8Small;

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
static int pick_bm(int64_t S, int E, int32_t w) {
  if (w == FG_E4M3) return use_big_tiles(S, E) ? GF8Big::BM : GF8Small::BM;
  return use_big_tiles(S, E) ? GBf16Big::BM : GBf16Small::BM;
}

static MoeLayout layout(const moe_desc& d) {
  MoeLayout L;
  L.S = d.T * d.top_k;
  L.BM = pick_bm(L.S, d.E, d.w_dtype);
  size_t o = 0;
  L.nblocks = (int)((d.T + ROUTE_TOKENS - 1) / ROUTE_TOKENS);
  L.tile_off = o;
  o = align_up(o + sizeof(int32_t) * (size_t)(d.E + 1));
  L.counts = o;
  o = align_up(o + sizeof(int32_t) * (size_t)L.nblocks * (size_t)d.E);
  L.h = o;
  o = align_up(o + (size_t)L.S * (size_t)d.I * 2);
  L.y = o;
  o = align_up(o + (size_t)L.S * (size_t)d.H * 4);
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

fg_status validate_desc(const moe_desc* d, const char* fn) {
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

// Resident workgroups of a kernel on the current device (occupancy × CUs),
// queried once per kernel and device. Concurrent first calls from several
// host threads compute the same value; the relaxed atomics keep that free
// of data races.
template <class TL, int EPI>
static int resident_workgroups() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cached[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_kernel<TL, EPI, false>, TL::THREADS, 0) !=
            hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
    v = per_cu * cus;
    cached[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// n-tiles: gate/up tiles cover BN/2 columns of h (BN weight rows, gate and
// up interleaved), down tiles BN columns of the output.

template <class TL, int EPI>
static hipError_t launch_grouped(GroupedArgs a, int64_t S, hipStream_t s) {
  a.tiles_n = EPI == EPI_GATEUP ? (int)((a.I + TL::BN / 2 - 1) / (TL::BN / 2)) : (int)((a.Nw + TL::BN - 1) / TL::BN);
  a.tiles_n_grid = (a.tiles_n + 7) / 8 * 8;
  // the m-tile count is known only on the device; its upper bound is
  // Σ_e ceil(n_e / BM) ≤ (S + E·(BM − 1)) / BM
  const int64_t mtiles = (S + (int64_t)a.E * (TL::BM - 1)) / TL::BM;
  const int64_t upper = mtiles * a.tiles_n_grid;
  // Small (decode) tiles stream weights: size the grid to the resident
  // workgroups so that no partial last wave of workgroups idles the chip.
  int64_t grid;
  if (TL::BM <= 32) {
    const int64_t res = resident_workgroups<TL, EPI>();
    grid = res < upper ? res : upper;
    grid = grid / 8 * 8 > 0 ? grid / 8 * 8 : 8;
  } else {
    // 8 ranges of at most ceil(real tiles / 8) entries each. bf16 tiles take
    // one entry per workgroup; e4m3 tiles run as many workgroups as are
    // resident (a multiple of 8), each taking every (G / 8)-th entry of its
    // range, so the m-tiles that share a weight tile start together in
    // every round (e4m3 step 666.5 vs 679.3 µs; bf16 937 vs 921 µs).
    grid = 8 * ((mtiles * a.tiles_n + 7) / 8);
    if constexpr (TL::IN == In::E4M3) {
      const int64_t res = resident_workgroups<TL, EPI>() / 8 * 8;
      if (res >= 8 && res < grid) grid = res;
    }
  }
  if constexpr (EPI == EPI_GATEUP) {
    // the token matrix: S / k rows of K elements
    const int64_t a_bytes = S / a.k * a.K * TL::ESIZE;
    if (a_bytes > ((int64_t)1 << 31))
      return launch(grouped_kernel<TL, EPI, true>, dim3((unsigned)grid), dim3(TL::THREADS), 0, s, a);
    a.a_bytes = static_cast<uint32_t>(a_bytes);
  }
  return launch(grouped_kernel<TL, EPI, false>, dim3((unsigned)grid), dim3(TL::THREADS), 0, s, a);
}

}  // namespace fg

using namespace fg;

extern "C" size_t moe_workspace_bytes(const moe_desc* d) {
  if (validate_desc(d, "moe_workspace_bytes") != FG_OK) return 0;
  return layout(*d).total;
}

// The MoE step on a given workspace (the body of both entry points):
// validates every argument, then enqueues the launches.
fg_status fg::moe_run(const char* fn, const moe_desc* d, const void* tokens, const float* router_logits,
                      const void* w_gateup, const void* w_down, const float* s_gateup, const float* s_down,
                      void* out, int32_t* topk_idx, float* topk_w, int32_t* perm, int32_t* expert_offsets,
                      void* workspace, size_t ws_bytes, void* stream) {
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
  Launches lc;
  if (T == 0) {
    // no tokens: every expert is empty (a fill kernel, not a memset node, so
    // that the call may be captured into a graph)
    lc.add(launch(fill_i32_kernel, dim3((unsigned)((d->E + 1 + 255) / 256)), dim3(256), 0, s, expert_offsets,
                  d->E + 1, 0));
    return check_launch(fn, lc);
  }
  const char* a_tokens = static_cast<const char*>(tokens);
  float* sx = reinterpret_cast<float*>(ws + L.sx);
  uint8_t* xq = f8 ? reinterpret_cast<uint8_t*>(ws + L.xq) : nullptr;
  const uint16_t* tok16 = static_cast<const uint16_t*>(tokens);
  if (f8) a_tokens = ws + L.xq;
  int32_t* counts = reinterpret_cast<int32_t*>(ws + L.counts);
  // with e4m3 the token quantisation rides in the routing launch: four rows
  // per block after the routing blocks
  const unsigned qblocks = f8 ? (unsigned)((d->T + 3) / 4) : 0u;
  if (L.nblocks == 1) {
    // one routing block, which also places the slots
    lc.add(launch(moe_route_kernel<true>, dim3(1 + qblocks), dim3(64 * ROUTE_WAVES), 0, s, router_logits, T, d->E,
                  d->top_k, topk_idx, topk_w, counts, L.BM, expert_offsets, tile_off, perm, tok16, d->H, xq, sx));
  } else {
    lc.add(launch(moe_route_kernel<false>, dim3((unsigned)L.nblocks + qblocks), dim3(64 * ROUTE_WAVES), 0, s,
                  router_logits, T, d->E, d->top_k, topk_idx, topk_w, counts, L.BM, expert_offsets, tile_off, perm,
                  tok16, d->H, xq, sx));
    lc.add(launch(moe_place_kernel, dim3((unsigned)L.nblocks), dim3(64 * PLACE_WAVES), 0, s, topk_idx, counts,
                  (int)S, d->E, d->top_k, L.nblocks, L.BM, expert_offsets, tile_off, perm));
  }

  GroupedArgs g{};
  g.perm = perm;
  g.offsets = expert_offsets;
  g.tile_off = tile_off;
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
  const bool big = use_big_tiles(S, d->E);
  if (f8)
    lc.add(big ? launch_grouped<GF8Big, EPI_GATEUP>(g, S, s) : launch_grouped<GF8Small, EPI_GATEUP>(g, S, s));
  else
    lc.add(big ? launch_grouped<GBf16Big, EPI_GATEUP>(g, S, s) : launch_grouped<GBf16Small, EPI_GATEUP>(g, S, s));

  // down: [S, I] × [H, I]ᵀ → y_slot [S, H] fp32, scattered to slot order (unweighted)
  const char* hA = ws + L.h;
  float* sh = reinterpret_cast<float*>(ws + L.sh);
  if (f8) {
    lc.add(launch(quantize_rows_kernel, dim3((unsigned)((S + 3) / 4)), dim3(256), 0, s,
                  reinterpret_cast<const uint16_t*>(ws + L.h), S, d->I, reinterpret_cast<uint8_t*>(ws + L.hq), sh));
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
  if (f8)
    lc.add(big ? launch_grouped<GF8Big, EPI_DOWN>(g, S, s) : launch_grouped<GF8Small, EPI_DOWN>(g, S, s));
  else
    lc.add(big ? launch_grouped<GBf16Big, EPI_DOWN>(g, S, s) : launch_grouped<GBf16Small, EPI_DOWN>(g, S, s));

  lc.add(launch_finalize(reinterpret_cast<const float*>(ws + L.y), topk_w, out, d->T, d->H, d->top_k, s));
  return check_launch(fn, lc);
}

extern "C" fg_status moe_grouped_ffn(const moe_desc* d, const void* tokens, const float* router_logits,
                                     const void* w_gateup, const void* w_down, const float* s_gateup,
                                     const float* s_down, void* out, int32_t* topk_idx, float* topk_w,
                                     int32_t* perm, int32_t* expert_offsets, void* workspace, size_t ws_bytes,
                                     void* stream) {
  clear_error();
  return moe_run("moe_grouped_ffn", d, tokens, router_logits, w_gateup, w_down, s_gateup, s_down, out, topk_idx,
                 topk_w, perm, expert_offsets, workspace, ws_bytes, stream);
}

extern "C" fg_status moe_finalize(const void* y_slot, void* out, int64_t T, int64_t H, int32_t top_k, void* stream) {
  clear_error();
  const char* fn = "moe_finalize";
  if (T < 0 || T > 0x7fffffffLL || H <= 0 || H > (1 << 20))
    return fail(FG_ERR_INVALID_ARG, "%s: bad T=%lld or H=%lld", fn, (long long)T, (long long)H);
  if (top_k < 1 || top_k > KMAX) return fail(FG_ERR_INVALID_ARG, "%s: top_k=%d outside 1..%d", fn, top_k, KMAX);
  if (H % 8 != 0) return fail(FG_ERR_ALIGNMENT, "%s: H must be a multiple of 8", fn);
  if (T == 0) return FG_OK;
  if (y_slot == nullptr || out == nullptr) return fail(FG_ERR_INVALID_ARG, "%s: NULL pointer", fn);
  if (!aligned16(y_slot) || !aligned16(out)) return fail(FG_ERR_ALIGNMENT, "%s: pointers must be 16-byte aligned", fn);
  Launches lc;
  lc.add(launch_finalize(static_cast<const uint16_t*>(y_slot), nullptr, out, T, H, top_k,
                         static_cast<hipStream_t>(stream)));
  return check_launch(fn, lc);
}
