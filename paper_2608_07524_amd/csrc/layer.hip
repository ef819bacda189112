// Element-wise and row-wise kernels of the transformer layer that wraps the
// attention kernels (the per-layer unit the profiling of Sec. 3.5 times and
// Eqs. (4)-(6) count): RMSNorm forward and backward, and the tanh form of
// GELU forward and backward.  All HBM-bound: one read and one write per
// element, 16-byte accesses, fp32 arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layer_launch.h"

namespace dcp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One wavefront per row of h values (h a multiple of 8): y = x * r * g with
// r = 1 / sqrt(mean(x^2) + eps); r is kept for the backward.
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const __bf16* __restrict__ x, const __bf16* __restrict__ g,
                                                          __bf16* __restrict__ y, float* __restrict__ rstd, int64_t rows,
                                                          int h, float eps) {
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const __bf16* xr = x + row * h;
  float ss = 0.f;
  for (int c = 8 * lane; c < h; c += 512) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(xr + c);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += float(v[e]) * float(v[e]);
  }
  const float r = rsqrtf(wave_sum(ss) / float(h) + eps);
  if (lane == 0) rstd[row] = r;
  for (int c = 8 * lane; c < h; c += 512) {
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(xr + c);
    const bf16x8 gv = *reinterpret_cast<const bf16x8*>(g + c);
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = __bf16(float(v[e]) * r * float(gv[e]));
    *reinterpret_cast<bf16x8*>(y + row * h + c) = o;
  }
}

// Backward of y = g * x * r for dy (fp32), plus a residual gradient:
//   dx = res + r * (g*dy - xh * mean(g*dy*xh)),  xh = x * r,
// and this block's partial sums of dg = sum_rows dy * xh (one row of
// `partial` per block; a second kernel adds the blocks in a fixed order, so
// the result is deterministic).  Each wavefront walks kNormBwdRows / 4 rows;
// a lane owns the columns 8*lane + 512*k (k < kNormMaxChunks, h <= 4096) and
// keeps their dg partials in registers until the block's end.
constexpr int kNormBwdRows = 16;  // rows per block (4 per wavefront): enough blocks to keep every CU busy
constexpr int kNormMaxChunks = 8;  // 16-byte column chunks per lane: h <= 64 * 8 * 8

__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(const float* __restrict__ dy, const __bf16* __restrict__ x,
                                                          const __bf16* __restrict__ g, const float* __restrict__ rstd,
                                                          const __bf16* __restrict__ res, __bf16* __restrict__ dx,
                                                          float* __restrict__ partial, int64_t rows, int h) {
  extern __shared__ float dg_lds[];  // [4 wavefronts][h]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float acc[kNormMaxChunks][8];
#pragma unroll
  for (int k = 0; k < kNormMaxChunks; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
  const int64_t r0 = int64_t(blockIdx.x) * kNormBwdRows + wave * (kNormBwdRows / 4);
  for (int i = 0; i < kNormBwdRows / 4; ++i) {
    const int64_t row = r0 + i;
    if (row >= rows) break;
    const float r = rstd[row];
    float dot = 0.f;
#pragma unroll
    for (int k = 0; k < kNormMaxChunks; ++k) {
      const int c = 8 * lane + 512 * k;
      if (c < h) {
        const bf16x8 xv = *reinterpret_cast<const bf16x8*>(x + row * h + c);
        const bf16x8 gv = *reinterpret_cast<const bf16x8*>(g + c);
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(dy + row * h + c);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(dy + row * h + c + 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = e < 4 ? d0[e] : d1[e - 4];
          const float xh = float(xv[e]) * r;
          dot += float(gv[e]) * d * xh;
          acc[k][e] += d * xh;
        }
      }
    }
    const float mean = wave_sum(dot) / float(h);
#pragma unroll
    for (int k = 0; k < kNormMaxChunks; ++k) {
      const int c = 8 * lane + 512 * k;
      if (c < h) {
        const bf16x8 xv = *reinterpret_cast<const bf16x8*>(x + row * h + c);
        const bf16x8 gv = *reinterpret_cast<const bf16x8*>(g + c);
        const bf16x8 rv = *reinterpret_cast<const bf16x8*>(res + row * h + c);
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(dy + row * h + c);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(dy + row * h + c + 4);
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = e < 4 ? d0[e] : d1[e - 4];
          o[e] = __bf16(float(rv[e]) + r * (float(gv[e]) * d - float(xv[e]) * r * mean));
        }
        *reinterpret_cast<bf16x8*>(dx + row * h + c) = o;
      }
    }
  }
  float* dgw = dg_lds + wave * h;
#pragma unroll
  for (int k = 0; k < kNormMaxChunks; ++k) {
    const int c = 8 * lane + 512 * k;
    if (c < h)
#pragma unroll
      for (int e = 0; e < 8; ++e) dgw[c + e] = acc[k][e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < h; c += 256)
    partial[int64_t(blockIdx.x) * h + c] = dg_lds[c] + dg_lds[h + c] + dg_lds[2 * h + c] + dg_lds[3 * h + c];
}

// dg[c] += sum over blocks of partial[b][c].  A workgroup takes 64 columns;
// its four wavefronts each sum every fourth partial row, then the four sums
// are added; the order is fixed, so the result is deterministic.
__global__ __launch_bounds__(256) void colsum_add_kernel(const float* __restrict__ partial, float* __restrict__ dg,
                                                         int nblocks, int h) {
  __shared__ float sums[4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = blockIdx.x * 64 + lane;
  // four independent running sums per lane (rows b = 16i + 4j + wave for j
  // = 0..3), so that loads overlap; added in a fixed order
  float s4[4] = {0.f, 0.f, 0.f, 0.f};
  if (c < h) {
    int b = wave;
    for (; b + 12 < nblocks; b += 16)
#pragma unroll
      for (int j = 0; j < 4; ++j) s4[j] += partial[int64_t(b + 4 * j) * h + c];
    for (int j = 0; b < nblocks; b += 4, ++j) s4[j & 3] += partial[int64_t(b) * h + c];
  }
  sums[wave][lane] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
  __syncthreads();
  if (wave == 0 && c < h) dg[c] += ((sums[0][lane] + sums[1][lane]) + sums[2][lane]) + sums[3][lane];
}

// GELU, tanh form: a = u/2 * (1 + tanh(k0 * (u + k1 u^3))).
constexpr float kGeluK0 = 0.7978845608028654f;  // sqrt(2 / pi)
constexpr float kGeluK1 = 0.044715f;

__global__ __launch_bounds__(256) void gelu_fwd_kernel(const __bf16* __restrict__ u, __bf16* __restrict__ a, int64_t n8) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n8) return;
  const bf16x8 v = reinterpret_cast<const bf16x8*>(u)[i];
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float x = float(v[e]);
    o[e] = __bf16(0.5f * x * (1.f + tanhf(kGeluK0 * (x + kGeluK1 * x * x * x))));
  }
  reinterpret_cast<bf16x8*>(a)[i] = o;
}

// du = da * d/du GELU(u) = da * (0.5 (1 + t) + 0.5 u (1 - t^2) k0 (1 + 3 k1 u^2)).
__global__ __launch_bounds__(256) void gelu_bwd_kernel(const __bf16* __restrict__ u, const __bf16* __restrict__ da,
                                                       __bf16* __restrict__ du, int64_t n8) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n8) return;
  const bf16x8 v = reinterpret_cast<const bf16x8*>(u)[i];
  const bf16x8 d = reinterpret_cast<const bf16x8*>(da)[i];
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float x = float(v[e]);
    const float t = tanhf(kGeluK0 * (x + kGeluK1 * x * x * x));
    const float dgelu = 0.5f * (1.f + t) + 0.5f * x * (1.f - t * t) * kGeluK0 * (1.f + 3.f * kGeluK1 * x * x);
    o[e] = __bf16(float(d[e]) * dgelu);
  }
  reinterpret_cast<bf16x8*>(du)[i] = o;
}

}  // namespace

hipError_t launch_rmsnorm_fwd(const void* x, const void* g, void* y, float* rstd, int64_t rows, int h, float eps,
                              hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_fwd_kernel, dim3(unsigned((rows + 3) / 4)), dim3(256), 0, s,
                     static_cast<const __bf16*>(x), static_cast<const __bf16*>(g), static_cast<__bf16*>(y), rstd, rows,
                     h, eps);
  return hipGetLastError();
}

int64_t rmsnorm_bwd_blocks(int64_t rows) { return (rows + kNormBwdRows - 1) / kNormBwdRows; }

hipError_t launch_rmsnorm_bwd(const float* dy, const void* x, const void* g, const float* rstd, const void* res,
                              void* dx, float* partial, float* dg, int64_t rows, int h, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int64_t nb = rmsnorm_bwd_blocks(rows);
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(unsigned(nb)), dim3(256), size_t(4) * h * sizeof(float), s, dy,
                     static_cast<const __bf16*>(x), static_cast<const __bf16*>(g), rstd,
                     static_cast<const __bf16*>(res), static_cast<__bf16*>(dx), partial, rows, h);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(colsum_add_kernel, dim3(unsigned((h + 63) / 64)), dim3(256), 0, s, partial, dg, int(nb), h);
  return hipGetLastError();
}

hipError_t launch_gelu_fwd(const void* u, void* a, int64_t n, hipStream_t s) {
  const int64_t n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  hipLaunchKernelGGL(gelu_fwd_kernel, dim3(unsigned((n8 + 255) / 256)), dim3(256), 0, s,
                     static_cast<const __bf16*>(u), static_cast<__bf16*>(a), n8);
  return hipGetLastError();
}

hipError_t launch_gelu_bwd(const void* u, const void* da, void* du, int64_t n, hipStream_t s) {
  const int64_t n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  hipLaunchKernelGGL(gelu_bwd_kernel, dim3(unsigned((n8 + 255) / 256)), dim3(256), 0, s,
                     static_cast<const __bf16*>(u), static_cast<const __bf16*>(da), static_cast<__bf16*>(du), n8);
  return hipGetLastError();
}

}  // namespace dcp
