// Host-side launch interface of the layer kernels (layer.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcp {

// y = x * rstd * g per row (bf16 [rows, h], h a multiple of 8); rstd fp32 [rows].
hipError_t launch_rmsnorm_fwd(const void* x, const void* g, void* y, float* rstd, int64_t rows, int h, float eps,
                              hipStream_t s);
// dx = res + RMSNorm backward of dy (fp32 [rows, h]); dg (fp32 [h]) += the
// gain gradient, reduced through `partial` (fp32 [rmsnorm_bwd_blocks(rows), h]).
hipError_t launch_rmsnorm_bwd(const float* dy, const void* x, const void* g, const float* rstd, const void* res,
                              void* dx, float* partial, float* dg, int64_t rows, int h, hipStream_t s);
int64_t rmsnorm_bwd_blocks(int64_t rows);
// a = GELU(u) and du = da * GELU'(u), n elements (a multiple of 8), bf16.
hipError_t launch_gelu_fwd(const void* u, void* a, int64_t n, hipStream_t s);
hipError_t launch_gelu_bwd(const void* u, const void* da, void* du, int64_t n, hipStream_t s);

}  // namespace dcp
