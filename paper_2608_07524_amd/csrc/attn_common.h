// Device-side building blocks for the CDNA4 (gfx950) attention kernels.
//
// Matrix-core conventions used throughout (v_mfma_f32_32x32x16_bf16, one
// 64-lane wavefront, lane = 32*g + i with g in {0,1}, i in [0,32)):
//   A operand (32 x 16): lane (g, i) holds row i, 8 contraction indices
//   B operand (16 x 32): lane (g, j) holds column j, the same 8 indices
//   C/D (32 x 32, fp32): lane (g, j), register r holds row
//                        8*(r/4) + 4*g + (r%4), column j.
// Which 8 contraction indices a lane holds only has to agree between A and
// B, so each kernel picks the assignment that makes its operands cheapest
// to fetch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tile_shapes.h"

namespace dcp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Bounds [lo, hi) of the sequence holding window offset x (0 <= x < n,
// the window's length), from the window's mask of sequence starts (bit 0
// is always set).
__device__ __forceinline__ void window_bounds(const uint64_t* __restrict__ starts, int x, int n, int& lo,
                                              int& hi) {
  lo = 0;
  hi = n;
#pragma unroll
  for (int w = 0; w < kWindowWords; ++w) {
    const uint64_t m = starts[w];
    const int r = x - 64 * w;  // x's bit in word w (outside 0..63 when x is in another word)
    const uint64_t upto = r < 0 ? 0ull : (r >= 63 ? ~0ull : (2ull << r) - 1);
    const uint64_t le = m & upto, gt = m & ~upto;  // starts at or before x, after x
    if (le) lo = 64 * w + 63 - __builtin_clzll(le);  // words ascend: the last hit is the nearest
    if (gt) hi = min(hi, 64 * w + __builtin_ctzll(gt));
  }
}

// Kernel-local lambdas are always inlined: a call would need a stack frame
// (scratch memory) and spill the caller's live registers around it.
#define DCP_INLINE __attribute__((always_inline))


// The dispatcher hands workgroup i to die i % 8.  Work lists are laid out
// as 8 consecutive per-die lists of `per_xcd` entries, so a die walks its
// own list in order and tiles that share K/V (or Q/dO) meet in its L2.
__device__ __forceinline__ const WorkUnit& unit_for_block(const WorkUnit* units, int per_xcd) {
  const int i = blockIdx.x;
  return units[(i % kNumXcd) * per_xcd + i / kNumXcd];
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16: lane (g4, i), g4 = lane / 16, holds row i of
// A (16 x 32) and column i of B (32 x 16) with the 8 contraction indices of
// group g4; C/D lane (g4, i), register r holds row 4*g4 + r, column i.
__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Wavefront issue priority around matrix-core phases: with two wavefronts
// on a SIMD, the one feeding the matrix cores issues first and the other
// fills the gaps with vector work.
__device__ __forceinline__ void mfma_prio_hi() { __builtin_amdgcn_s_setprio(1); }
__device__ __forceinline__ void mfma_prio_lo() { __builtin_amdgcn_s_setprio(0); }

// Max / sum of a value with the lane 32 positions away (the two halves of a
// wavefront), via the gfx950 cross-half lane swap.
__device__ __forceinline__ float half_swap_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Transposing LDS read of 16-bit data (gfx950 ds_read_b64_tr_b16).  Within
// each group of 16 lanes, lane t names 4 consecutive elements; lane i gets
// element (i % 4) of the rows named by lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4.
// With lane t pointing at row (t / 4), columns 4*(t % 4) .. +3 of a
// row-major tile, lane i receives column i of 4 consecutive rows.
__device__ __forceinline__ bf16x4 lds_read_tr(const __bf16* p) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ bf16x8 cat(const bf16x4& lo, const bf16x4& hi) {
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

__device__ __forceinline__ bf16x8 lds_read_b128(const __bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// The same reads through LDS-address-space (32-bit) pointers.  Indexing a
// __shared__ array through lds_ptr() keeps the address arithmetic in 32
// bits, so constant terms fold into the instructions' offset fields.
#define DCP_LDS __attribute__((address_space(3)))
typedef DCP_LDS __bf16 lds_bf16;
typedef DCP_LDS float lds_f32;
template <typename T>
__device__ __forceinline__ DCP_LDS T* lds_ptr(T* p) {
  return (DCP_LDS T*)(p);
}
__device__ __forceinline__ bf16x4 lds_read_tr(const lds_bf16* p) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((DCP_LDS i16x4*)(p)));
}
__device__ __forceinline__ bf16x8 lds_read_b128(const lds_bf16* p) { return *(const DCP_LDS bf16x8*)(p); }
__device__ __forceinline__ f32x4 lds_read_f32x4(const lds_f32* p) { return *(const DCP_LDS f32x4*)(p); }

// Waits until at most N vector-memory operations of this wavefront are in
// flight (gfx9 s_waitcnt: vmcnt split over bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their maxima, i.e. not waited on).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// Direct global -> LDS copy of one ROWS-row tile (gfx950
// global_load_lds_dwordx4: each lane moves 16 bytes, a wavefront fills 64
// consecutive 16-byte LDS slots, no registers involved).  In LDS, slot
// (r, c) of the tile sits at byte 16*(r*CPR_PAD + c); slots c < CPR_DATA of
// rows r < valid_rows come from src + r*row_stride + 8c, slot c == CPR_DATA
// from `first_pad` (a 16-byte constant chunk, e.g. [1, 0, ..., 0] for a
// row-sum column) and every other slot from `zero`.  The tile occupies
// ELEMS = 512*NINS elements (plus the group skews below): when ROWS*CPR_PAD is not a multiple of 64,
// the last copy also fills the slots past the tile with zeros.  Every
// wavefront issues exactly NI instructions per tile (the last one repeated
// when they do not split evenly; the repeat rewrites identical bytes), so
// a fixed wait_vmcnt count covers the tile on every wavefront.  Completion
// is tracked by vmcnt only: wait, then barrier, before reading the tile.
// GSKEW > 0 starts every 16-row group of the tile GSKEW elements further
// on (row r at element r * 8 * CPR_PAD + GSKEW * (r / 16)): a group is a
// whole number of copies, so only the copies' LDS bases move.
template <int ROWS, int CPR_PAD, int CPR_DATA, int NW, int GSKEW = 0>
struct DmaTile {
  static constexpr int NSLOT = ROWS * CPR_PAD;
  static constexpr int NINS = (NSLOT + 63) / 64;
  static constexpr int NI = (NINS + NW - 1) / NW;
  static constexpr int IPG = GSKEW ? 16 * CPR_PAD / 64 : 1;  // copies per 16-row group
  static_assert(GSKEW == 0 || (16 * CPR_PAD % 64 == 0 && ROWS % 16 == 0), "skewed groups are whole copies");
  static constexpr int ELEMS = 512 * NINS + GSKEW * (NINS / IPG);
  static_assert(CPR_DATA < CPR_PAD, "pad slots hold the constant chunks");
  // element offset of copy t inside the tile
  __device__ __forceinline__ static constexpr int dst(int t) { return 512 * t + GSKEW * (t / IPG); }

  __device__ __forceinline__ static void issue(__bf16* lds_tile, const __bf16* src, int64_t row_stride,
                                               int valid_rows, const __bf16* zero, const __bf16* first_pad,
                                               int wave, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const int slot = 64 * t + lane;
      const int r = slot / CPR_PAD, c = slot % CPR_PAD;
      const __bf16* g = zero;
      if (c < CPR_DATA) {
        if (r < valid_rows && r < ROWS) g = src + int64_t(r) * row_stride + 8 * c;
      } else if (c == CPR_DATA && r < ROWS) {
        g = first_pad;
      }
      dma16(g, lds_tile + dst(t));
    }
  }

  // Full tiles (every row inside the sequence): this lane's byte offsets
  // from the tile's first row, one per copy it issues.  Slot (r, c) reads
  // chunk c of row r when c < CPR_DATA and chunk 0 of the same row
  // otherwise (such columns are either multiplied by zero register
  // operands or produce output columns that are never stored); slots past
  // the tile repeat its last row.  The offsets do not change from tile to
  // tile, so a full tile's copies take no vector arithmetic.
  struct FullOffsets {
    uint32_t off[NI];
  };
  __device__ __forceinline__ static FullOffsets full_offsets(int64_t row_stride, int wave, int lane) {
    FullOffsets fo;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const int slot = 64 * t + lane;
      const int r = min(slot / CPR_PAD, ROWS - 1), c = slot % CPR_PAD;
      fo.off[i] = uint32_t((int64_t(r) * row_stride + 8 * (c < CPR_DATA ? c : 0)) * 2);
    }
    return fo;
  }
  // Copies a full tile whose first row is at `src` (wavefront-uniform):
  // scalar base plus the precomputed offsets (global_load_lds_dwordx4 in
  // its scalar-base form).
  __device__ __forceinline__ static void issue_full(__bf16* lds_tile, const __bf16* src, const FullOffsets& fo,
                                                    int wave) {
    // (readfirstlane returns a signed int: both halves go through uint32_t
    // so the low word is zero-extended, never sign-extended into the high one)
    const uint64_t a = reinterpret_cast<uint64_t>(src);
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32)));
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a)));
    const uint64_t base = (uint64_t(hi) << 32) | uint64_t(lo);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const uint32_t m0 = __builtin_amdgcn_readfirstlane(
          static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_tile + dst(t))));
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                   :
                   : "s"(m0), "v"(fo.off[i]), "s"(base)
                   : "memory");
    }
  }

  // As issue_full, but slot column SKIP of every row is left untouched
  // (its lanes are masked off), so a constant written there once stays.
  template <int SKIP>
  struct SkipMasks {
    uint64_t m[NI];
  };
  template <int SKIP>
  __device__ __forceinline__ static SkipMasks<SKIP> skip_masks(int wave, int lane) {
    SkipMasks<SKIP> sm;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const int slot = 64 * t + lane;
      sm.m[i] = __builtin_amdgcn_ballot_w64(slot % CPR_PAD != SKIP || slot / CPR_PAD >= ROWS);
    }
    return sm;
  }
  template <int SKIP>
  __device__ __forceinline__ static void issue_full_skip(__bf16* lds_tile, const __bf16* src, const FullOffsets& fo,
                                                         const SkipMasks<SKIP>& sm, int wave) {
    const uint64_t a = reinterpret_cast<uint64_t>(src);
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32)));
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a)));
    const uint64_t base = (uint64_t(hi) << 32) | uint64_t(lo);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const uint32_t m0 = __builtin_amdgcn_readfirstlane(
          static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_tile + dst(t))));
      uint64_t saved;
      asm volatile(
          "s_mov_b64 %0, exec\n\t"
          "s_mov_b64 exec, %1\n\t"
          "s_mov_b32 m0, %2\n\t"
          "global_load_lds_dwordx4 %3, %4\n\t"
          "s_mov_b64 exec, %0"
          : "=&s"(saved)
          : "s"(sm.m[i]), "s"(m0), "v"(fo.off[i]), "s"(base)
          : "memory");
    }
  }

  // One global_load_lds_dwordx4: lane i's 16 bytes at `g` land in LDS at
  // `lds_base` + 16*i.  Written as inline assembly: the compiler would
  // otherwise treat the copy as possibly aliasing every LDS read and wait
  // for it right away, which defeats copying ahead.  The callers' explicit
  // vmcnt waits and barriers order it instead; callers also settle their
  // own earlier vector loads before the first copy, so that no wait the
  // compiler inserts later stands for a load it tracks.  M0 is written here
  // and used by nothing else in these kernels (checked in the generated
  // code: no other M0 reader).
  __device__ __forceinline__ static void dma16(const __bf16* g, __bf16* lds_base) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_base)));  // low 32 bits = LDS offset
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(m0), "v"(reinterpret_cast<uint64_t>(g))
                 : "memory");
  }
};

// Direct global -> LDS copy of two N-element fp32 vectors stored back to
// back (gfx9 global_load_lds_dword: each lane moves 4 bytes, a wavefront
// fills 256 consecutive LDS bytes).  Element e < valid of the first vector
// comes from a[e], of the second from b[e]; every other element from the
// 4-byte constant at fill_a / fill_b.  Like DmaTile, every wavefront
// issues exactly NI instructions.
template <int N, int NW>
struct DmaVecPair {
  static constexpr int NINS = 2 * N / 64;
  static constexpr int NI = (NINS + NW - 1) / NW;
  static_assert(2 * N % 64 == 0, "vectors must fill whole wavefront copies");

  __device__ __forceinline__ static void issue(float* lds_vec, const float* a, const float* b, int valid,
                                               const float* fill_a, const float* fill_b, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = min(wave + NW * i, NINS - 1);
      const int e = 64 * t + lane;
      const bool second = e >= N;
      const int idx = second ? e - N : e;
      const float* g = idx < valid ? (second ? b : a) + idx : (second ? fill_b : fill_a);
      const uint32_t m0 = __builtin_amdgcn_readfirstlane(
          static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_vec + 64 * t)));
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off"
                   :
                   : "s"(m0), "v"(reinterpret_cast<uint64_t>(g))
                   : "memory");
    }
  }
};


}  // namespace dcp
