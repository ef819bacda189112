// Host-side launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tile_shapes.h"

namespace dcp {

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  const void* consts;  // device: the 16-byte constant chunks (workspace head)
  const void* units;   // device WorkUnit[n_units + n_wunits]: sequence tiles, then packed windows,
                       // each part 8 per-die lists
  const void* window_starts;  // device: 4 uint64 per packed window
  int n_units;
  int n_wunits;
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
  float* ndelta;          // fp32 [H, T] workspace: -rowsum(dO o O)
  float* lse2;            // fp32 [H, T] workspace: LSE * log2(e)
  const void* consts;     // device: the 16-byte constant chunks (workspace head)
  const void* units;      // device WorkUnit[n_units + n_wunits], key tiles then packed windows
  const void* window_starts;   // device: 4 uint64 per packed window of the key-tile list
  int n_units;
  int n_wunits;
  const void* qunits;     // device WorkUnit[n_qunits + n_wqunits], query tiles then packed windows
  const void* qwindow_starts;  // device: the same for the query-tile list
  int n_qunits;
  int n_wqunits;
  int rows_end;           // cu_seqlens[n]: rows past it are not touched
  int n_heads;
  int head_dim;
  int total_tokens;
  float scale;
  int causal;
  hipStream_t stream;
};

// Optional events recorded around the main attention kernel of each call
// (set through dcp_set_kernel_events; null when unused).
struct KernelEvents {
  hipEvent_t begin = nullptr;
  hipEvent_t end = nullptr;
};
KernelEvents& kernel_events();

hipError_t launch_fwd(const FwdArgs& a);
hipError_t launch_bwd(const BwdArgs& a);

// Fills n bf16 values with a deterministic pseudo-random pattern in
// [-1, 1) (used to give profiling runs realistic, finite inputs).
hipError_t launch_fill_bf16(void* p, int64_t n, uint32_t seed, hipStream_t stream);

}  // namespace dcp
