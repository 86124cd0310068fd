// rope.hip — QKV bias + rotary position embedding + paged KV-cache write of
// one decode step (paper §IV-A, "Bias + RoPE + KV update" in Table I).
//
// One workgroup per token. Every thread owns one work item of the token's
// row (more only when a row has more items than 1024 threads): for a
// half-split head a pair of 8-value chunks (c, c + D/16), whose values pair
// element by element; for an interleaved head one chunk (four adjacent
// pairs); for a value head one chunk, copied with its bias. A thread first
// issues its item's 16-byte loads (qkv and bias); while they are in flight
// the first D/2 threads compute the token's rotation factors (cos φ_i,
// sin φ_i), φ_i = pos·base^(−2i/D), with the angle formed and reduced in
// fp64 — it grows to ~10^5 rad at long positions, where an fp32 angle would
// already be off by ~10^-2 — and leave them in LDS as fp32. After one
// barrier each thread adds the bias, rotates in fp32 and stores 16 bytes at
// a time into q_out or the token's cache row. The cache row is resolved once
// per workgroup from the block table; tokens whose position or block id is
// out of range skip the cache stores.
#include <hip/hip_runtime.h>
#include <math.h>

#include "fg_host.hpp"
#include "fg_tile.hpp"
#include "fgemm.h"

namespace fg {

constexpr int ROPE_MAX_D = 256;

struct RopeArgs {
  const uint16_t* qkv;
  const uint16_t* bias;      // may be null
  const int32_t* positions;
  const int32_t* block_table;
  uint16_t* q_out;
  uint16_t* cache;
  int n_q, n_kv, D, bs, max_blocks;
  int64_t num_blocks;
  int width;                 // (n_q + 2·n_kv)·D
  int interleaved;
  int items_per_head;        // rotated items per head
  int rot_items, items;      // rotated items, all items of a token
  double log2_base;
};

__device__ __forceinline__ void unpack_bf16x8(const i32x4& v, float (&f)[8]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f[2 * q] = bf16_bits_to_f32((uint16_t)(v[q] & 0xffff));
    f[2 * q + 1] = bf16_bits_to_f32((uint16_t)((uint32_t)v[q] >> 16));
  }
}

__device__ __forceinline__ i32x4 pack_bf16x8(const float (&f)[8]) {
  i32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    o[q] = (int)((uint32_t)f32_to_bf16_bits(f[2 * q]) | ((uint32_t)f32_to_bf16_bits(f[2 * q + 1]) << 16));
  return o;
}

// The raw 16-byte chunks of one work item: the row chunk(s) and the matching
// bias chunk(s). Loaded before the rotation table exists, so that the first
// item's memory latency overlaps the table's computation.
struct ItemData {
  i32x4 x0, x1, b0, b1;
};

__device__ __forceinline__ i32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const i32x4*>(p); }

// Row element offsets of item `it`: e0 (and e1, the partner chunk of a
// half-split item). Value items have e1 unused.
__device__ __forceinline__ void item_offsets(const RopeArgs& a, int it, int& h, int& c, int& e0, int& e1) {
  if (it < a.rot_items) {
    h = it / a.items_per_head;
    c = it % a.items_per_head;
    e0 = h * a.D + c * 8;
    e1 = e0 + (a.D >> 1);
  } else {
    const int cpr = a.D / 8, vi = it - a.rot_items;
    h = vi / cpr;
    c = vi % cpr;
    e0 = (a.n_q + a.n_kv + h) * a.D + c * 8;
    e1 = e0;
  }
}

__device__ __forceinline__ ItemData load_item(const RopeArgs& a, const uint16_t* row, int it) {
  int h, c, e0, e1;
  item_offsets(a, it, h, c, e0, e1);
  const bool pair = it < a.rot_items && !a.interleaved;
  const i32x4 z = {0, 0, 0, 0};
  ItemData d;
  d.x0 = ld16(row + e0);
  d.x1 = pair ? ld16(row + e1) : z;
  d.b0 = a.bias != nullptr ? ld16(a.bias + e0) : z;
  d.b1 = pair && a.bias != nullptr ? ld16(a.bias + e1) : z;
  return d;
}

// Bias add, rotation (query and key items) and the stores of item `it`.
__device__ __forceinline__ void finish_item(const RopeArgs& a, const float (&cs)[2][ROPE_MAX_D / 2], int t,
                                            int64_t kv0, int it, const ItemData& d) {
  int h, c, e0, e1;
  item_offsets(a, it, h, c, e0, e1);
  const int half = a.D >> 1;
  const int64_t head_stride = (int64_t)a.bs * a.D;     // between heads of one cache row
  float x[8], bx[8];
  unpack_bf16x8(d.x0, x);
  unpack_bf16x8(d.b0, bx);
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] += bx[j];
  if (it >= a.rot_items) {
    if (kv0 < 0) return;
    uint16_t* dst = a.cache + kv0 + (int64_t)(a.n_kv + h) * head_stride;
    *reinterpret_cast<i32x4*>(dst + c * 8) = pack_bf16x8(x);
    return;
  }
  uint16_t* dst;
  if (h < a.n_q) {
    dst = a.q_out + ((int64_t)t * a.n_q + h) * a.D;
  } else {
    if (kv0 < 0) return;
    dst = a.cache + kv0 + (int64_t)(h - a.n_q) * head_stride;
  }
  if (!a.interleaved) {
    float y[8], by[8];
    unpack_bf16x8(d.x1, y);
    unpack_bf16x8(d.b1, by);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float co = cs[0][c * 8 + j], si = cs[1][c * 8 + j];
      const float u = x[j], w = y[j] + by[j];
      x[j] = u * co - w * si;
      y[j] = u * si + w * co;
    }
    *reinterpret_cast<i32x4*>(dst + c * 8) = pack_bf16x8(x);
    *reinterpret_cast<i32x4*>(dst + half + c * 8) = pack_bf16x8(y);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float co = cs[0][c * 4 + j], si = cs[1][c * 4 + j];
      const float u = x[2 * j], w = x[2 * j + 1];
      x[2 * j] = u * co - w * si;
      x[2 * j + 1] = u * si + w * co;
    }
    *reinterpret_cast<i32x4*>(dst + c * 8) = pack_bf16x8(x);
  }
}

// Rotation angle of pair i at position pos, reduced to [−π, π] in fp64
// (pos·θ_i reaches ~10^5 rad; 2π is split in two parts so that k·2π is
// exact to well below an fp32 ulp of the remainder), then sine and cosine in
// fp32 on the reduced argument.
__device__ __forceinline__ void rope_factor(int pos, int i, int D, double log2_base, float& co, float& si) {
  const double ang = (double)pos * exp2(-(double)(2 * i) / (double)D * log2_base);
  const double k = rint(ang * 0.15915494309189535);                 // 1/(2π)
  double r = fma(-k, 6.283185307179586, ang);                          // 2π, high part
  r = fma(-k, 2.4492935982947064e-16, r);                              // 2π − high part
  sincosf((float)r, &si, &co);
}

__global__ __launch_bounds__(1024) void bias_rope_kv_kernel(RopeArgs a) {
  __shared__ float cs[2][ROPE_MAX_D / 2];
  const int t = blockIdx.x;
  const uint16_t* row = a.qkv + (int64_t)t * a.width;
  const int first = threadIdx.x;
  ItemData d0;
  if (first < a.items) d0 = load_item(a, row, first);
  const int pos = a.positions[t];
  // element offset of cache[blk, 0, 0, r, 0], or −1 when the token writes no cache row
  int64_t kv0 = -1;
  if (pos >= 0 && pos / a.bs < a.max_blocks) {
    const int blk = a.block_table[(int64_t)t * a.max_blocks + pos / a.bs];
    if (blk >= 0 && (int64_t)blk < a.num_blocks) kv0 = ((int64_t)blk * 2 * a.n_kv * a.bs + pos % a.bs) * a.D;
  }
  for (int i = threadIdx.x; i < (a.D >> 1); i += blockDim.x) rope_factor(pos, i, a.D, a.log2_base, cs[0][i], cs[1][i]);
  __syncthreads();
  if (first < a.items) finish_item(a, cs, t, kv0, first, d0);
  for (int it = first + blockDim.x; it < a.items; it += blockDim.x) finish_item(a, cs, t, kv0, it, load_item(a, row, it));
}

}  // namespace fg

using namespace fg;

extern "C" fg_status bias_rope_kv_update(const rope_desc* d, const void* qkv, const void* bias,
                                         const int32_t* positions, const int32_t* block_table, void* q_out,
                                         void* kv_cache, void* stream) {
  clear_error();
  const char* fn = "bias_rope_kv_update";
  if (d == nullptr) return fail(FG_ERR_INVALID_ARG, "%s: desc is NULL", fn);
  const int64_t LIM = 0x7fffffffLL;
  if (d->T < 0 || d->T > LIM) return fail(FG_ERR_INVALID_ARG, "%s: bad T=%lld", fn, (long long)d->T);
  if (d->n_q_heads < 1 || d->n_kv_heads < 1 || d->n_q_heads > 4096 || d->n_kv_heads > 4096)
    return fail(FG_ERR_INVALID_ARG, "%s: head counts must be 1 .. 4096 (n_q=%d, n_kv=%d)", fn, d->n_q_heads,
                d->n_kv_heads);
  if (d->head_dim < 16) return fail(FG_ERR_INVALID_ARG, "%s: head_dim=%d below 16", fn, d->head_dim);
  if (d->head_dim % 16 != 0) return fail(FG_ERR_ALIGNMENT, "%s: head_dim=%d not a multiple of 16", fn, d->head_dim);
  if (d->head_dim > ROPE_MAX_D)
    return fail(FG_ERR_UNSUPPORTED, "%s: head_dim=%d above %d", fn, d->head_dim, ROPE_MAX_D);
  if (d->block_size < 1 || d->max_blocks < 1 || d->num_blocks < 1 || d->num_blocks > LIM)
    return fail(FG_ERR_INVALID_ARG, "%s: bad cache geometry (block_size=%d, max_blocks=%d, num_blocks=%lld)", fn,
                d->block_size, d->max_blocks, (long long)d->num_blocks);
  if ((double)d->num_blocks * 2.0 * d->n_kv_heads * d->block_size * d->head_dim > 4.0e18)
    return fail(FG_ERR_INVALID_ARG, "%s: cache of more than 2^62 elements", fn);
  if (!(d->rope_base > 0.0f) || !isfinite(d->rope_base))
    return fail(FG_ERR_INVALID_ARG, "%s: rope_base must be finite and > 0", fn);
  if (d->interleaved != 0 && d->interleaved != 1) return fail(FG_ERR_INVALID_ARG, "%s: interleaved must be 0 or 1", fn);
  if (d->T == 0) return FG_OK;
  if (qkv == nullptr || positions == nullptr || block_table == nullptr || q_out == nullptr || kv_cache == nullptr)
    return fail(FG_ERR_INVALID_ARG, "%s: NULL pointer", fn);
  if (!aligned16(qkv) || !aligned16(q_out) || !aligned16(kv_cache) || (bias != nullptr && !aligned16(bias)) ||
      (reinterpret_cast<uintptr_t>(positions) & 3u) != 0 || (reinterpret_cast<uintptr_t>(block_table) & 3u) != 0)
    return fail(FG_ERR_ALIGNMENT, "%s: bf16 pointers must be 16-byte and int32 pointers 4-byte aligned", fn);
  RopeArgs a;
  a.qkv = static_cast<const uint16_t*>(qkv);
  a.bias = static_cast<const uint16_t*>(bias);
  a.positions = positions;
  a.block_table = block_table;
  a.q_out = static_cast<uint16_t*>(q_out);
  a.cache = static_cast<uint16_t*>(kv_cache);
  a.n_q = d->n_q_heads;
  a.n_kv = d->n_kv_heads;
  a.D = d->head_dim;
  a.bs = d->block_size;
  a.max_blocks = d->max_blocks;
  a.num_blocks = d->num_blocks;
  a.width = (a.n_q + 2 * a.n_kv) * a.D;
  a.interleaved = d->interleaved;
  a.items_per_head = a.interleaved ? a.D / 8 : a.D / 16;
  a.rot_items = (a.n_q + a.n_kv) * a.items_per_head;
  a.items = a.rot_items + a.n_kv * (a.D / 8);
  a.log2_base = log2((double)d->rope_base);
  int threads = (a.items + 63) / 64 * 64;
  if (threads > 1024) threads = 1024;
  Launches lc;
  lc.add(launch(bias_rope_kv_kernel, dim3((unsigned)d->T), dim3(threads), 0, static_cast<hipStream_t>(stream), a));
  return check_launch(fn, lc);
}
