// Host-side launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcp {

// Query rows per forward workgroup: 4 wavefronts x 32 x kFwdNQB.
constexpr int kFwdNQB = 2;
// Key rows per backward workgroup (4 wavefronts x 32) and query rows per
// backward inner step.
constexpr int kBwdBN = 128;
constexpr int kBwdBM = 64;

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  const void* units;  // device WorkUnit[n_units]
  int n_units;
  int n_heads;
  int head_dim;
  int total_tokens;
  float scale;
  int causal;
  hipStream_t stream;
};

struct BwdArgs {
  const void* dout;
  const void* o;
  const float* lse;
  const void* q;
  const void* k;
  const void* v;
  void* dq;
  void* dk;
  void* dv;
  float* dq_acc;          // fp32 [T, H, D] workspace
  float* delta;           // fp32 [H, T] workspace
  const void* units;      // device WorkUnit[n_units], key tiles of kBwdBN rows
  int n_units;
  int rows_end;           // cu_seqlens[n]: rows past it are not touched
  int n_heads;
  int head_dim;
  int total_tokens;
  float scale;
  int causal;
  hipStream_t stream;
};

int fwd_tile_rows(int head_dim);
hipError_t launch_fwd(const FwdArgs& a);
hipError_t launch_bwd(const BwdArgs& a);

// Fills n bf16 values with a deterministic pseudo-random pattern in
// [-1, 1) (used to give profiling runs realistic, finite inputs).
hipError_t launch_fill_bf16(void* p, int64_t n, uint32_t seed, hipStream_t stream);

}  // namespace dcp
