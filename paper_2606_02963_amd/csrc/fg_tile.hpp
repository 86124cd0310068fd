// fg_tile.hpp — the tiled MFMA main loop shared by every GEMM in the library.
//
// One workgroup of WM × WN wave64s computes a BM × BN tile of acc = A·Bᵀ, where A rows and B rows are both contiguous along K (x rows and
// nn.Linear weight rows). Per K stage each tile row contributes 128 bytes
// (8 chunks of 16 B): 32 fp32, 64 bf16 or 128 e4m3 values. Stages are staged
// HBM → VGPR → LDS with 128-bit loads and stores and double-buffered in LDS,
// so the global loads of stage k+1 are in flight while stage k feeds the
// matrix cores. Inside LDS each row's chunk c is stored at chunk c ^ (row & 7)
// so that both the row-wise writes and the column-of-rows fragment reads hit
// eight distinct 16-byte bank groups.
//
// Fragments use the 16 × 16 MFMA shapes of gfx950 (wave64):
//   bf16  v_mfma_f32_16x16x32_bf16          (two per stage per fragment pair)
//   e4m3  v_mfma_scale_f32_16x16x128_f8f6f4 (one per stage, unit scales)
//   fp32  v_mfma_f32_16x16x4_f32            (eight per stage)
// For all three, lane l supplies row (l & 15) of the A block and column
// (l & 15) of the B block, and receives C[4·(l >> 4) + i][l & 15], i = 0..3.
// Which k each (lane group, register element) carries is the same function
// for A and B, so a lane may feed any fixed bijection of the stage's k values:
// lane group g = l >> 4 always reads chunks 2g and 2g + 1 (32 contiguous
// bytes) of its row, which keeps every fragment read a pair of 128-bit LDS
// reads for every input type.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

enum class In { F32, BF16, E4M3 };

template <In IN> struct InTraits;
template <> struct InTraits<In::F32>  { static constexpr int EPC = 4,  ESIZE = 4; };
template <> struct InTraits<In::BF16> { static constexpr int EPC = 8,  ESIZE = 2; };
template <> struct InTraits<In::E4M3> { static constexpr int EPC = 16, ESIZE = 1; };

template <In IN_, int BM_, int BN_, int WM_ = 2, int WN_ = 2>
struct Tile {
  static constexpr In IN = IN_;
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int WM = WM_, WN = WN_, NWAVES = WM * WN, THREADS = 64 * NWAVES;
  static constexpr int RSTRIDE = THREADS / 8;          // rows between a thread's successive loads
  static constexpr int TM = BM / WM, TN = BN / WN;     // wave tile
  static constexpr int FM = TM / 16, FN = TN / 16;     // 16×16 fragments per wave
  static constexpr int ROWB = 128;                      // bytes per tile row per stage
  static constexpr int EPC = InTraits<IN>::EPC;
  static constexpr int ESIZE = InTraits<IN>::ESIZE;
  static constexpr int BK = (ROWB / 16) * EPC;          // K elements per stage
  static constexpr int A_LD = BM * 8 / THREADS;         // 16-byte chunks per thread per stage
  static constexpr int B_LD = BN * 8 / THREADS;
  static constexpr int STAGE_BYTES = (BM + BN) * ROWB;
  static constexpr int LOOP_LDS = 2 * STAGE_BYTES;
  static_assert(BM % RSTRIDE == 0 && BN % RSTRIDE == 0, "tile sides must be multiples of THREADS/8");
  static_assert(TM % 16 == 0 && TN % 16 == 0, "wave tiles must be multiples of 16");
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ (row & 7)) << 4);
}

// Row sources for the stage loads. Thread t owns tile rows
// (t >> 3) + (THREADS/8)·p, p < NLD; `ptr[p]` is the start of that row in global
// memory. Rows past the matrix edge point at any valid row: their LDS copy
// only feeds accumulator rows / columns that are never stored.
template <int NLD>
struct RowSet {
  const char* ptr[NLD];
};

// Direct HBM → LDS load of one full stage (every row has 128 valid bytes at
// kbyte): global_load_lds_dwordx4 writes lane i's 16 bytes at LDS offset
// 16·i of a wave-uniform 1 KiB block, i.e. block b = wave + NWAVES·p holds
// tile rows 8b .. 8b + 7 with physical chunk i & 7. The lane therefore
// fetches logical chunk (i & 7) ^ (i >> 3), the inverse of the LDS swizzle.
template <int NWAVES, int NLD>
__device__ __forceinline__ void load_stage_direct(const RowSet<NLD>& rs, int64_t kbyte, char* sbase) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = (lane & 7) ^ (lane >> 3);
#pragma unroll
  for (int p = 0; p < NLD; ++p) {
    const char* src = rs.ptr[p] + kbyte + c * 16;
    char* dst = sbase + (wave + NWAVES * p) * 1024;
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(src),
                                     (__attribute__((address_space(3))) void*)(dst), 16, 0, 0);
  }
}

// Zero-filling load of a partial stage through VGPRs: chunks at or past
// kbytes read as zero, so the tail contributes nothing beyond K.
template <int RSTRIDE, int NLD>
__device__ __forceinline__ void load_stage_tail(const RowSet<NLD>& rs, int64_t kbyte, int64_t kbytes,
                                                char* sbase) {
  const int c = threadIdx.x & 7;
  const int r0 = threadIdx.x >> 3;
  const int64_t off = kbyte + c * 16;
#pragma unroll
  for (int p = 0; p < NLD; ++p) {
    i32x4 v = {0, 0, 0, 0};
    if (off < kbytes) v = *reinterpret_cast<const i32x4*>(rs.ptr[p] + off);
    *reinterpret_cast<i32x4*>(sbase + lds_off(r0 + RSTRIDE * p, c)) = v;
  }
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// acc[fm][fn] += A-fragments × B-fragments for one LDS stage.
template <class TL>
__device__ __forceinline__ void mma_stage(const char* sA, const char* sB, int wm, int wn,
                                          f32x4 (&acc)[TL::FM][TL::FN]) {
  const int l = threadIdx.x & 63;
  const int g = l >> 4;
  const int r16 = l & 15;
  if constexpr (TL::IN == In::BF16) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 af[TL::FM], bfr[TL::FN];
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm) {
        const int r = wm * TL::TM + fm * 16 + r16;
        af[fm] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const i32x4*>(sA + lds_off(r, 2 * g + h)));
      }
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) {
        const int r = wn * TL::TN + fn * 16 + r16;
        bfr[fn] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const i32x4*>(sB + lds_off(r, 2 * g + h)));
      }
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < TL::FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[fm], bfr[fn], acc[fm][fn], 0, 0, 0);
    }
  } else if constexpr (TL::IN == In::E4M3) {
    i32x8 af[TL::FM], bfr[TL::FN];
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm) {
      const int r = wm * TL::TM + fm * 16 + r16;
      const i32x4 lo = *reinterpret_cast<const i32x4*>(sA + lds_off(r, 2 * g));
      const i32x4 hi = *reinterpret_cast<const i32x4*>(sA + lds_off(r, 2 * g + 1));
      af[fm] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) {
      const int r = wn * TL::TN + fn * 16 + r16;
      const i32x4 lo = *reinterpret_cast<const i32x4*>(sB + lds_off(r, 2 * g));
      const i32x4 hi = *reinterpret_cast<const i32x4*>(sB + lds_off(r, 2 * g + 1));
      bfr[fn] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        // operand formats 0 = FP8 E4M3 for A and B; E8M0 scale 127 = 2^0
        acc[fm][fn] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
            af[fm], bfr[fn], acc[fm][fn], 0, 0, 0, 127, 0, 127);
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      f32x4 af[TL::FM], bfr[TL::FN];
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm) {
        const int r = wm * TL::TM + fm * 16 + r16;
        af[fm] = __builtin_bit_cast(f32x4, *reinterpret_cast<const i32x4*>(sA + lds_off(r, 2 * g + h)));
      }
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) {
        const int r = wn * TL::TN + fn * 16 + r16;
        bfr[fn] = __builtin_bit_cast(f32x4, *reinterpret_cast<const i32x4*>(sB + lds_off(r, 2 * g + h)));
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < TL::FN; ++fn)
            acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[fm][s], bfr[fn][s], acc[fm][fn], 0, 0, 0);
    }
  }
}

// The K loop: acc = Σ_k A[rows]·B[rows]ᵀ over kbytes bytes of each row.
// `lds` must hold TL::LOOP_LDS bytes. A partial last stage (kbytes not a
// multiple of 128) is loaded first through the zero-filling path; the full
// stages then stream through the two LDS buffers with direct loads, the
// loads of stage s + 1 in flight while stage s is multiplied. Ends with a
// barrier, so the caller may reuse the LDS immediately.
template <class TL>
__device__ __forceinline__ void gemm_mainloop(const RowSet<TL::A_LD>& ra, const RowSet<TL::B_LD>& rb,
                                              int64_t kbytes, char* lds,
                                              f32x4 (&acc)[TL::FM][TL::FN]) {
  const int wave = threadIdx.x >> 6;
  const int wm = wave / TL::WN, wn = wave % TL::WN;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) acc[fm][fn] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t KT = kbytes / TL::ROWB;   // full stages
  if (kbytes % TL::ROWB != 0) {
    char* sb = lds + TL::STAGE_BYTES;
    load_stage_tail<TL::RSTRIDE, TL::A_LD>(ra, KT * TL::ROWB, kbytes, sb);
    load_stage_tail<TL::RSTRIDE, TL::B_LD>(rb, KT * TL::ROWB, kbytes, sb + TL::BM * TL::ROWB);
    __syncthreads();
    mma_stage<TL>(sb, sb + TL::BM * TL::ROWB, wm, wn, acc);
    __syncthreads();
  }
  if (KT == 0) return;
  load_stage_direct<TL::NWAVES, TL::A_LD>(ra, 0, lds);
  load_stage_direct<TL::NWAVES, TL::B_LD>(rb, 0, lds + TL::BM * TL::ROWB);
  wait_vmem();
  __syncthreads();
  for (int64_t kt = 0; kt < KT; ++kt) {
    char* cur = lds + (kt & 1) * TL::STAGE_BYTES;
    char* nxt = lds + ((kt + 1) & 1) * TL::STAGE_BYTES;
    if (kt + 1 < KT) {
      load_stage_direct<TL::NWAVES, TL::A_LD>(ra, (kt + 1) * TL::ROWB, nxt);
      load_stage_direct<TL::NWAVES, TL::B_LD>(rb, (kt + 1) * TL::ROWB, nxt + TL::BM * TL::ROWB);
    }
    mma_stage<TL>(cur, cur + TL::BM * TL::ROWB, wm, wn, acc);
    wait_vmem();
    __syncthreads();
  }
}

// Position of accumulator element (fm, fn, i) inside the workgroup tile.
template <class TL>
__device__ __forceinline__ int acc_row(int fm, int i) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  return (wave / TL::WN) * TL::TM + fm * 16 + 4 * (l >> 4) + i;
}
template <class TL>
__device__ __forceinline__ int acc_col(int fn) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  return (wave % TL::WN) * TL::TN + fn * 16 + (l & 15);
}

// fp32 → bf16 bits with round-to-nearest-even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float v) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// Reduce over the 16 lanes that share a tile row (lanes with equal l >> 4).
__device__ __forceinline__ float row16_sum(float v) {
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

// Stage the tile through LDS and write it with 16-byte row-contiguous stores.
// `vals(fm, fn, i, v, c)` returns whether accumulator element (fm, fn, i)
// is stored and, if so, its fp32 value v (converted to bf16 here) and its
// output column c within the OUTC-column output tile; `row_ptr(r)` gives the
// destination of tile row r (nullptr to skip it) and `ncols` the number of
// valid output columns (a multiple of 8). `lds` needs BM·(2·OUTC + 16) bytes; a barrier is
// taken before the writes and after the reads.
template <class TL, int OUTC, class Vals, class RowPtr>
__device__ __forceinline__ void store_tile_bf16(char* lds, Vals vals, RowPtr row_ptr, int ncols) {
  constexpr int PITCH = OUTC * 2 + 16;
  __syncthreads();
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v;
        int c;
        if (vals(fm, fn, i, v, c)) {
          const int r = acc_row<TL>(fm, i);
          *reinterpret_cast<uint16_t*>(lds + r * PITCH + c * 2) = f32_to_bf16_bits(v);
        }
      }
  __syncthreads();
  constexpr int CPR = OUTC / 8;  // 16-byte chunks per row
  constexpr int TOTAL = TL::BM * CPR;
  for (int idx = threadIdx.x; idx < TOTAL; idx += TL::THREADS) {
    const int r = idx / CPR, c = idx % CPR;
    char* dst = row_ptr(r);
    if (dst != nullptr && c * 8 < ncols)
      *reinterpret_cast<i32x4*>(dst + c * 16) = *reinterpret_cast<const i32x4*>(lds + r * PITCH + c * 16);
  }
}

}  // namespace fg
