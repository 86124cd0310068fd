// fg_tile.hpp — the tiled MFMA main loop shared by every GEMM in the library.
//
// One workgroup of WM × WN wave64s computes a BM × BN tile of acc = A·Bᵀ,
// where A rows and B rows are both contiguous along K (x rows and nn.Linear
// weight rows). Per K stage each tile row contributes 128 bytes (8 chunks of
// 16 B): 32 fp32, 64 bf16 or 128 e4m3 values. Stages go from memory straight
// into LDS (buffer / global loads with the LDS bit, 16 bytes per lane) and
// are double-buffered there, so the loads of stage k+1 are in flight while
// stage k feeds the matrix cores (staging through VGPRs and 128-bit LDS
// writes measured slower). Inside LDS each row's chunk c is stored at chunk
// c ^ (row & 7) ^ ((row >> 3) & 1): a fragment read (16 consecutive rows, one
// chunk) then touches sixteen distinct 16-byte bank groups of the 64-bank
// LDS (rows alternate between its two 128-byte halves; the eight rows of one
// parity land on eight distinct chunks), and any eight consecutive rows also
// stay distinct, while the row-wise writes remain contiguous.
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

// PRIO_: raise the wave priority (s_setprio 1) over each substep's MFMA and
// fragment-read cluster, so that with two workgroups per compute unit a wave
// that has matrix work ready issues it ahead of the other workgroup's loads
// and barrier waits.
template <In IN_, int BM_, int BN_, int WM_ = 2, int WN_ = 2, bool PRIO_ = false>
struct Tile {
  static constexpr In IN = IN_;
  static constexpr bool PRIO = PRIO_;
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
  return row * 128 + ((chunk ^ (row & 7) ^ ((row >> 3) & 1)) << 4);
}

// Row sources for the stage loads. Thread t owns tile rows
// r = (t >> 3) + (THREADS/8)·p, p < NLD. Two sources implement the same two
// operations:
//   stage(kbyte, sbase)        direct HBM → LDS load of one full stage;
//   tail(kbyte, kbytes, sbase) zero-filling load of a partial last stage.
// The direct loads write lane i's 16 bytes at LDS offset 16·i of a
// wave-uniform 1 KiB block, i.e. block b = wave + NWAVES·p holds tile rows
// 8b .. 8b + 7 with physical chunk i & 7; the lane therefore fetches logical
// chunk (i & 7) ^ (i >> 3) ^ (b & 1), the inverse of the LDS swizzle. NWAVES
// is even, so b & 1 = wave & 1 for every p.

// Gathered rows (MoE token rows through the permutation): one pointer per
// owned row, for matrices of more than 2^31 bytes (the MoE kernels gather
// smaller ones through a buffer descriptor). Rows past the matrix edge point
// at any valid row: their LDS copy only feeds accumulator rows / columns
// that are never stored.
template <int NLD>
struct RowSet {
  const char* ptr[NLD];

  template <int NWAVES>
  __device__ __forceinline__ void stage(int64_t kbyte, char* sbase) const {
    static_assert(NWAVES % 2 == 0, "the fetched chunk assumes an even wave count");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = (lane & 7) ^ (lane >> 3) ^ (wave & 1);
#pragma unroll
    for (int p = 0; p < NLD; ++p) {
      const char* src = ptr[p] + kbyte + c * 16;
      char* dst = sbase + (wave + NWAVES * p) * 1024;
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(src),
                                       (__attribute__((address_space(3))) void*)(dst), 16, 0, 0);
    }
  }

  // Every load is issued before the first LDS write (global address space,
  // so the compiler need not order them after the writes): one memory round
  // trip. Chunks past kbytes load the row's first chunk and are replaced by
  // zeros.
  template <int RSTRIDE>
  __device__ __forceinline__ void tail(int64_t kbyte, int64_t kbytes, char* sbase) const {
    typedef const __attribute__((address_space(1))) i32x4 GlobalChunk;
    const int c = threadIdx.x & 7;
    const int r0 = threadIdx.x >> 3;
    const int64_t off = kbyte + c * 16;
    const bool in = off < kbytes;
    i32x4 v[NLD];
#pragma unroll
    for (int p = 0; p < NLD; ++p) v[p] = *(GlobalChunk*)(ptr[p] + (in ? off : 0));
#pragma unroll
    for (int p = 0; p < NLD; ++p)
      *reinterpret_cast<i32x4*>(sbase + lds_off(r0 + RSTRIDE * p, c)) = in ? v[p] : i32x4{0, 0, 0, 0};
  }
};

// Buffer-resource loads (MUBUF with the LDS bit, and a 128-bit MUBUF load for
// the tail), bound to the LLVM intrinsics. Offsets beyond num_records read
// as zero, which is how rows past the matrix edge are filled.
__device__ void fg_raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) void* lds, uint32_t size,
                                       uint32_t voffset, uint32_t soffset, uint32_t offset,
                                       uint32_t aux) __asm("llvm.amdgcn.raw.buffer.load.lds");
__device__ i32x4 fg_raw_buffer_load_b128(i32x4 rsrc, uint32_t voffset, uint32_t soffset,
                                         uint32_t aux) __asm("llvm.amdgcn.raw.buffer.load.v4i32");
__device__ void fg_raw_buffer_store_b128(i32x4 data, i32x4 rsrc, uint32_t voffset, uint32_t soffset,
                                         uint32_t aux) __asm("llvm.amdgcn.raw.buffer.store.v4i32");
// Cache-policy bit of the buffer intrinsics that makes an access device
// coherent (sc1 on gfx950: a store writes through to the device coherence
// point, a load does not hit a stale line), as for agent-scope atomics.
constexpr uint32_t FG_CPOL_DEVICE = 16;

// 128-bit buffer descriptor: 48-bit base, stride 0 (raw), num_records bytes,
// and the data-format word used for untyped raw access on gfx9-class parts.
__device__ __forceinline__ i32x4 make_buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return i32x4{static_cast<int>(static_cast<uint32_t>(b)), static_cast<int>(static_cast<uint32_t>(b >> 32) & 0xffff),
               static_cast<int>(bytes), 0x00020000};
}

// Strided rows (dense x and W tiles, MoE weight rows): the rows a lane loads
// lie at a fixed byte step (pstride) from its first one (rowoff0) inside one
// buffer descriptor, so each lane keeps one 32-bit offset instead of NLD
// pointers. Offsets at or beyond the descriptor's size read as zero, which
// is how rows past the matrix edge are filled. Every offset stays below
// 2^31 (the plans bound the tile's byte span).
template <int NLD, int RSTRIDE>
struct BufRows {
  i32x4 rsrc;         // wave-uniform
  uint32_t voff;      // rowoff0 + 16·(fetched chunk)
  uint32_t pstride;   // bytes between a lane's successive rows
  uint32_t rowoff0;   // byte offset of a lane's first row

  // Tile rows r = (t >> 3) + RSTRIDE·p of a matrix whose rows are
  // row_stride bytes apart; rows at or past rows_valid read as zero.
  __device__ __forceinline__ void init(const char* base, int64_t rows_valid, int64_t rows_tile, int64_t row_stride) {
    const int64_t rows = rows_valid < rows_tile ? rows_valid : rows_tile;
    init_rows(base, static_cast<uint32_t>(rows * row_stride), static_cast<uint32_t>(threadIdx.x >> 3) *
              static_cast<uint32_t>(row_stride), static_cast<uint32_t>(RSTRIDE * row_stride));
  }

  // A lane's rows at byte offsets first + pstride·p from `base`; bytes
  // at or past `bytes` read as zero. `base` and `bytes` must be uniform
  // across the wave.
  __device__ __forceinline__ void init_rows(const char* base, uint32_t bytes, uint32_t first, uint32_t step) {
    const i32x4 r = make_buffer_rsrc(base, bytes);
    rsrc = i32x4{__builtin_amdgcn_readfirstlane(r[0]), __builtin_amdgcn_readfirstlane(r[1]),
                 __builtin_amdgcn_readfirstlane(r[2]), __builtin_amdgcn_readfirstlane(r[3])};
    pstride = step;
    rowoff0 = first;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    voff = first + static_cast<uint32_t>(((lane & 7) ^ (lane >> 3) ^ (wave & 1)) * 16);
  }

  template <int NWAVES>
  __device__ __forceinline__ void stage(int64_t kbyte, char* sbase) const {
    static_assert(NWAVES % 2 == 0, "the fetched chunk assumes an even wave count");
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int p = 0; p < NLD; ++p) {
      char* dst = sbase + (wave + NWAVES * p) * 1024;
      fg_raw_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(dst), 16,
                             voff + p * pstride + static_cast<uint32_t>(kbyte), 0, 0, 0);
    }
  }

  // Every load is issued before the first LDS write (one memory round trip);
  // chunks past kbytes get an out-of-range offset and read as zero.
  template <int RS>
  __device__ __forceinline__ void tail(int64_t kbyte, int64_t kbytes, char* sbase) const {
    const int c = threadIdx.x & 7;
    const int r0 = threadIdx.x >> 3;
    const int64_t off = kbyte + c * 16;
    const uint32_t rowoff = rowoff0 + static_cast<uint32_t>(off);
    const bool in = off < kbytes;
    i32x4 v[NLD];
#pragma unroll
    for (int p = 0; p < NLD; ++p) v[p] = fg_raw_buffer_load_b128(rsrc, in ? rowoff + p * pstride : 0x80000000u, 0, 0);
#pragma unroll
    for (int p = 0; p < NLD; ++p) *reinterpret_cast<i32x4*>(sbase + lds_off(r0 + RS * p, c)) = v[p];
  }
};

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Operand fragments of one substep. A stage is split into SUB substeps:
// bf16 and fp32 take chunk 2g + h in substep h (h = 0, 1), so one substep is
// one 16×16×32 bf16 MFMA (or four 16×16×4 fp32 MFMAs) per fragment pair;
// e4m3 needs both chunks 2g, 2g + 1 for its single 16×16×128 MFMA, so its
// stage is one substep.
template <class TL, In IN = TL::IN> struct Frag;
template <class TL> struct Frag<TL, In::BF16> { static constexpr int SUB = 2; using V = bf16x8; V a[TL::FM], b[TL::FN]; };
template <class TL> struct Frag<TL, In::F32>  { static constexpr int SUB = 2; using V = f32x4; V a[TL::FM], b[TL::FN]; };
template <class TL> struct Frag<TL, In::E4M3> { static constexpr int SUB = 1; using V = i32x8; V a[TL::FM], b[TL::FN]; };

template <class TL>
__device__ __forceinline__ i32x4 lds16(const char* stage, int row, int chunk) {
  return *reinterpret_cast<const i32x4*>(stage + lds_off(row, chunk));
}

// Read substep h of the stage at `sA` (B rows follow the BM A rows).
template <class TL>
__device__ __forceinline__ void read_frag(const char* sA, int wm, int wn, int h, Frag<TL>& F) {
  const char* sB = sA + TL::BM * TL::ROWB;
  const int l = threadIdx.x & 63;
  const int g = l >> 4, r16 = l & 15;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm) {
    const int r = wm * TL::TM + fm * 16 + r16;
    if constexpr (TL::IN == In::E4M3) {
      const i32x4 lo = lds16<TL>(sA, r, 2 * g), hi = lds16<TL>(sA, r, 2 * g + 1);
      F.a[fm] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    } else {
      F.a[fm] = __builtin_bit_cast(typename Frag<TL>::V, lds16<TL>(sA, r, 2 * g + h));
    }
  }
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int r = wn * TL::TN + fn * 16 + r16;
    if constexpr (TL::IN == In::E4M3) {
      const i32x4 lo = lds16<TL>(sB, r, 2 * g), hi = lds16<TL>(sB, r, 2 * g + 1);
      F.b[fn] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    } else {
      F.b[fn] = __builtin_bit_cast(typename Frag<TL>::V, lds16<TL>(sB, r, 2 * g + h));
    }
  }
}

// acc[fm][fn] += A-fragment × B-fragment for one substep.
template <class TL>
__device__ __forceinline__ void mma_frag(const Frag<TL>& F, f32x4 (&acc)[TL::FM][TL::FN]) {
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) {
      if constexpr (TL::IN == In::BF16) {
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.a[fm], F.b[fn], acc[fm][fn], 0, 0, 0);
      } else if constexpr (TL::IN == In::E4M3) {
        // operand formats 0 = FP8 E4M3 for A and B; E8M0 scale 127 = 2^0
        acc[fm][fn] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(F.a[fm], F.b[fn], acc[fm][fn], 0, 0,
                                                                       0, 127, 0, 127);
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x4f32(F.a[fm][s], F.b[fn][s], acc[fm][fn], 0, 0, 0);
      }
    }
}

// Issue order inside a substep: each LDS read of the next substep's
// fragments goes out right after one MFMA of the current substep, so the
// reads stream while the matrix core works instead of waiting as one block.
template <class TL>
__device__ __forceinline__ void interleave_reads_with_mfma() {
  constexpr int NRD = (TL::FM + TL::FN) * (TL::IN == In::E4M3 ? 2 : 1);
  constexpr int NMF = TL::FM * TL::FN * (TL::IN == In::F32 ? 4 : 1);
  constexpr int PAIRS = NRD < NMF ? NRD : NMF;
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
  }
  if constexpr (NMF > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, NMF - PAIRS, 0);
}

// One substep of the pipelined loop: substep j is in Fc; prepare substep
// j + 1 in Fn, then multiply Fc. When j + 1 opens stage s = (j + 1) / SUB,
// the workgroup first waits for stage s to have landed (its loads were
// issued one stage earlier), synchronises — which also retires every read of
// stage s − 1 — and issues the direct loads of stage s + 1 into the buffer
// stage s − 1 used. Loads past the last stage repeat the last stage into
// that free buffer, which is never read again: the loop body needs no branch.
// A wave that is not LIVE only loads and synchronises.
template <class TL, bool LIVE, class LA, class LB>
__device__ __forceinline__ void pipelined_substep(int64_t j, int64_t KT, const LA& ra, const LB& rb,
                                                  char* lds, int wm, int wn, const Frag<TL>& Fc, Frag<TL>& Fn,
                                                  f32x4 (&acc)[TL::FM][TL::FN]) {
  constexpr int SUB = Frag<TL>::SUB;
  const int64_t nx = j + 1;
  const int64_t s = nx / SUB;
  const int h = static_cast<int>(nx % SUB);
  if (h == 0) {
    wait_vmem();
    __syncthreads();
    const int64_t sl = s + 1 < KT ? s + 1 : KT - 1;
    char* dst = lds + ((s + 1) & 1) * TL::STAGE_BYTES;
    ra.template stage<TL::NWAVES>(sl * TL::ROWB, dst);
    rb.template stage<TL::NWAVES>(sl * TL::ROWB, dst + TL::BM * TL::ROWB);
  }
  if constexpr (LIVE) {
    if constexpr (TL::PRIO) __builtin_amdgcn_s_setprio(1);
    read_frag<TL>(lds + (s & 1) * TL::STAGE_BYTES, wm, wn, h, Fn);
    mma_frag<TL>(Fc, acc);
    interleave_reads_with_mfma<TL>();
    if constexpr (TL::PRIO) __builtin_amdgcn_s_setprio(0);
  }
}

// The K loop after its first loads (see gemm_mainloop); LIVE = false runs
// the same loads and barriers without fragment reads or MFMAs.
template <class TL, bool LIVE, class LA, class LB>
__device__ __forceinline__ void mainloop_stages(const LA& ra, const LB& rb, int64_t KT, char* lds, int wm, int wn,
                                                f32x4 (&acc)[TL::FM][TL::FN]) {
  constexpr int SUB = Frag<TL>::SUB;
  Frag<TL> F0, F1;
  if constexpr (SUB == 1 && TL::FM * TL::FN > 8) {
    // large e4m3 tiles: one substep per stage and 32-byte fragments; a
    // second fragment set would not fit beside two resident workgroups, so
    // each wave reads and multiplies in turn and the other workgroup's waves
    // fill the gaps. (Small e4m3 tiles take the pipelined loop below, with
    // one stage per substep.)
    for (int64_t kt = 0; kt < KT; ++kt) {
      if constexpr (LIVE) {
        read_frag<TL>(lds + (kt & 1) * TL::STAGE_BYTES, wm, wn, 0, F0);
        mma_frag<TL>(F0, acc);
      }
      wait_vmem();
      __syncthreads();
      const int64_t sl = kt + 2 < KT ? kt + 2 : KT - 1;
      char* dst = lds + (kt & 1) * TL::STAGE_BYTES;
      ra.template stage<TL::NWAVES>(sl * TL::ROWB, dst);
      rb.template stage<TL::NWAVES>(sl * TL::ROWB, dst + TL::BM * TL::ROWB);
    }
  } else {
    if constexpr (LIVE) read_frag<TL>(lds, wm, wn, 0, F0);
    const int64_t J = KT * SUB;               // substeps
    int64_t j = 0;
    for (; j + 2 < J; j += 2) {
      pipelined_substep<TL, LIVE>(j, KT, ra, rb, lds, wm, wn, F0, F1, acc);
      pipelined_substep<TL, LIVE>(j + 1, KT, ra, rb, lds, wm, wn, F1, F0, acc);
    }
    // the last one or two substeps: multiply F0 before reading the final
    // substep into the same registers (one fragment set live, not two, beside
    // the accumulators); if the final substep opens the last stage its loads
    // were issued long ago, so only the barrier is needed
    if constexpr (LIVE) mma_frag<TL>(F0, acc);
    if (J - j == 2) {
      const int64_t s = (j + 1) / SUB;
      const int h = static_cast<int>((j + 1) % SUB);
      if (h == 0) {
        wait_vmem();
        __syncthreads();
      }
      if constexpr (LIVE) {
        read_frag<TL>(lds + (s & 1) * TL::STAGE_BYTES, wm, wn, h, F0);
        mma_frag<TL>(F0, acc);
      }
    }
  }
}

// The K loop: acc = Σ_k A[rows]·B[rows]ᵀ over kbytes bytes of each row.
// `lds` must hold TL::LOOP_LDS bytes. A partial last stage (kbytes not a
// multiple of 128) is loaded first through the zero-filling path; the full
// stages then stream through the two LDS buffers, each stage's direct loads
// in flight while the stage before it is multiplied (the large e4m3 tiles
// issue stage s + 2 into the buffer stage s has just been read from), and
// the fragments of substep j + 1 are read during the MFMAs of substep j. Ends with a
// barrier, so the caller may reuse the LDS immediately. A wave whose A rows
// all lie at or past `rows_valid` (a ragged last row tile; wave-uniform)
// only takes part in the loads and barriers: it reads no fragments and
// issues no MFMAs, which leaves its SIMD to the other waves; its
// accumulators stay zero.
template <class TL, class LA, class LB>
__device__ __forceinline__ void gemm_mainloop(const LA& ra, const LB& rb,
                                              int64_t kbytes, char* lds,
                                              f32x4 (&acc)[TL::FM][TL::FN], int rows_valid = TL::BM) {
  constexpr int SUB = Frag<TL>::SUB;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / TL::WN, wn = wave % TL::WN;
  const bool live = __builtin_amdgcn_readfirstlane(wm * TL::TM < rows_valid ? 1 : 0) != 0;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) acc[fm][fn] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t KT = kbytes / TL::ROWB;   // full stages
  if (KT > 0) {
    ra.template stage<TL::NWAVES>(0, lds);
    rb.template stage<TL::NWAVES>(0, lds + TL::BM * TL::ROWB);
  }
  if (kbytes % TL::ROWB != 0) {
    // the partial last stage goes through buffer 1 while stage 0 lands in
    // buffer 0: both requests are in flight together
    char* sb = lds + TL::STAGE_BYTES;
    ra.template tail<TL::RSTRIDE>(KT * TL::ROWB, kbytes, sb);
    rb.template tail<TL::RSTRIDE>(KT * TL::ROWB, kbytes, sb + TL::BM * TL::ROWB);
    __syncthreads();
    if (live) {
      Frag<TL> F;
#pragma unroll
      for (int h = 0; h < SUB; ++h) {
        read_frag<TL>(sb, wm, wn, h, F);
        mma_frag<TL>(F, acc);
      }
    }
    __syncthreads();
  }
  if (KT == 0) return;
  if (KT > 1) {
    char* s1 = lds + TL::STAGE_BYTES;
    ra.template stage<TL::NWAVES>(TL::ROWB, s1);
    rb.template stage<TL::NWAVES>(TL::ROWB, s1 + TL::BM * TL::ROWB);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(TL::A_LD + TL::B_LD) : "memory");
  } else {
    wait_vmem();
  }
  __syncthreads();
  if (live)
    mainloop_stages<TL, true>(ra, rb, KT, lds, wm, wn, acc);
  else
    mainloop_stages<TL, false>(ra, rb, KT, lds, wm, wn, acc);
  wait_vmem();
  __syncthreads();
}

// K-slice exchange of one output tile computed by `ks` workgroups, each over
// a slice of K (split-K). Every slice stores its partial accumulator tile
// with device-coherent (sc1) 16-byte stores (thread-major, so each wave's
// stores are contiguous), waits until they are acknowledged and then counts
// its arrival in the tile's 64-bit counter word (high half: the run's
// epoch, low half: arrivals in that run) with an atomic compare-and-swap. An
// arrival that finds another epoch — left by an earlier run, or whatever the
// workspace held — starts the count at 1 for this run, so the workspace
// needs no initialisation. The slice that brings the count to ks reads the
// partials back with device-coherent loads and adds them in slice order (so
// the sum does not depend on which slice arrives last), resets the count to
// 0 under the same epoch (a captured graph replaying the launch with the
// same epoch then starts clean) and returns true; the others return false.
// Only the partials and the counter are shared, and both are accessed
// device-coherently, so no cache-wide write-back or invalidation is needed.
// `partials` holds ks partial tiles of FM·FN·THREADS 16-byte values; `flag`
// is one word of LDS.
template <class TL>
__device__ __forceinline__ bool slice_gather(f32x4 (&acc)[TL::FM][TL::FN], f32x4* partials, int ks, int slice,
                                             unsigned long long* counter, unsigned epoch, unsigned* flag) {
  constexpr int NF = TL::FM * TL::FN;
  constexpr uint32_t SLICE = NF * TL::THREADS * 16;   // bytes of one partial tile
  const int tid = threadIdx.x;
  const i32x4 rsrc = make_buffer_rsrc(partials, static_cast<uint32_t>(ks) * SLICE);
  const uint32_t lane_off = static_cast<uint32_t>(tid) * 16;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn)
      fg_raw_buffer_store_b128(__builtin_bit_cast(i32x4, acc[fm][fn]), rsrc,
                               slice * SLICE + (fm * TL::FN + fn) * TL::THREADS * 16 + lane_off, 0, FG_CPOL_DEVICE);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const unsigned long long ep = (unsigned long long)epoch << 32;
    unsigned long long old = __hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), want;
    while (true) {
      want = (old & 0xffffffff00000000ull) == ep ? old + 1 : ep | 1ull;
      if (__hip_atomic_compare_exchange_strong(counter, &old, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT))
        break;
    }
    *flag = (unsigned)want;
  }
  __syncthreads();
  if (*flag != (unsigned)ks) return false;
  // read back one fragment row (FN loads) at a time: the memory clobber keeps
  // the compiler from hoisting every load, whose destinations would not fit
  // beside the accumulators
#pragma unroll 1
  for (int k = slice == 0 ? 1 : 0; k < ks; ++k) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm) {
      f32x4 v[TL::FN];
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        v[fn] = __builtin_bit_cast(
            f32x4, fg_raw_buffer_load_b128(rsrc, k * SLICE + (fm * TL::FN + fn) * TL::THREADS * 16 + lane_off, 0,
                                           FG_CPOL_DEVICE));
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) {
        if (k == 0)
          acc[fm][fn] = v[fn];
        else
          acc[fm][fn] += v[fn];
      }
      asm volatile("" ::: "memory");
    }
  }
  if (tid == 0) __hip_atomic_store(counter, (unsigned long long)epoch << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return true;
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

// Reduce over the 16 lanes that share a tile row (lanes with equal l >> 4,
// one DPP row). Four DPP steps: lane ^ 1 and lane ^ 2 (quad permutes) give
// every lane its quad's total, then rotations of the row by 4 and by 8 add
// the other three quads. The maximum is the same in all 16 lanes; a sum may
// differ in the last bit between lanes (different association), so callers
// take lane (l & 15) == 0's value.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x124>(v);  // row_ror:4
  v += dpp_f<0x128>(v);  // row_ror:8
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x124>(v));
  v = fmaxf(v, dpp_f<0x128>(v));
  return v;
}

// Native-instruction math for the tails (v_exp_f32 = 2^x, v_rcp_f32,
// v_rsq_f32; each within a few ulp of fp32, far inside the bf16 and fp32
// output tolerances). e^x = 2^(x·log2 e) underflows to 0 below about −87
// and overflows to +inf above about 88, which the callers rely on.
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fast_rsqrt(float x) { return __builtin_amdgcn_rsqf(x); }
// σ(x) = 1/(1 + e^−x): 1 for large x, 0 (through rcp(+inf)) for very negative x.
__device__ __forceinline__ float fast_sigmoid(float x) { return fast_rcp(1.0f + fast_exp(-x)); }

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
