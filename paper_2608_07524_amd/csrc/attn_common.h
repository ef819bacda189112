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

namespace dcp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// One tile of work: rows [row0, row0 + rows) of the packed tensor, all in
// the sequence that occupies rows [seq0, seq0 + seqlen).
struct WorkUnit {
  int32_t row0;
  int32_t rows;
  int32_t seq0;
  int32_t seqlen;
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

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

__device__ __forceinline__ void atomic_add_f32(float* p, float v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace dcp
