// Measurement probe (not part of libdcp): the bf16 matrix-core rate that
// chains of dependent 32x32x16 products reach with nothing else running,
// two wavefronts per SIMD on every CU -- the practical ceiling the attention
// kernels' product rates are compared with (the published dense peak
// assumes every clock at the nominal engine clock).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;  // per workgroup: two per SIMD

template <int kChains>
__global__ __launch_bounds__(64 * kWaves, 1) void mfma_rate_kernel(float* __restrict__ out, int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = __bf16(float((lane + i) % 7) * 0.125f);
    b[i] = __bf16(float((lane * 3 + i) % 5) * 0.0625f);
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[size_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

}  // namespace

// Launches `blocks` workgroups of 8 wavefronts, each wavefront running
// `iters` rounds of `chains` (1, 2 or 4) independent 32x32x16 bf16 products
// (each round extends every chain by one dependent product), on `stream`;
// `out` holds blocks * 512 floats.  Returns the flops the launch performs
// (blocks * 8 * iters * chains * 32768) through *flops, and 0, -1 for bad
// arguments, or the launch error code.
extern "C" int dcp_probe_mfma_rate(float* out, int blocks, int iters, int chains, void* stream, double* flops) {
  if (!out || !flops || blocks <= 0 || iters <= 0 || (chains != 1 && chains != 2 && chains != 4)) return -1;
  const dim3 grid{unsigned(blocks), 1, 1}, block{64 * kWaves, 1, 1};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (chains == 1) hipLaunchKernelGGL(mfma_rate_kernel<1>, grid, block, 0, s, out, iters);
  if (chains == 2) hipLaunchKernelGGL(mfma_rate_kernel<2>, grid, block, 0, s, out, iters);
  if (chains == 4) hipLaunchKernelGGL(mfma_rate_kernel<4>, grid, block, 0, s, out, iters);
  *flops = double(blocks) * kWaves * double(iters) * chains * 32768.0;
  return int(hipGetLastError());
}
