// Host-side launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcp {

// Query rows per forward workgroup: kFwdWaves wavefronts x 32.
constexpr int kFwdWaves = 8;
// Backward, dK/dV pass: `waves` wavefronts per workgroup, each owning
// 32*kb keys whose K, V fragments and dK, dV accumulators stay resident,
// stepping over `bm` queries at a time through a `stages`-deep LDS ring;
// waves_per_eu is the occupancy the register allocation must allow.
// Head widths up to 72 run two wavefronts of 32 keys per SIMD, with Q and
// dO held once per ring stage (the transposing reads of dV and dK use the
// row-read copy, at the cost of some bank conflicts), which leaves LDS for
// a four-stage ring of 64-query tiles.  At head width 128 the resident
// state needs more than the 256 registers two wavefronts per SIMD could
// each have, so that width runs one wavefront per SIMD; its ring holds Q
// and dO once too, in two stages of 128-query tiles (139 KB of the 160 KB
// of LDS), so that a barrier comes every four 32-query blocks.
// dQ pass: kBwdDqWaves wavefronts of 32 queries, kBwdDqBN keys per step,
// K held once per ring stage (its transposing reads share the row-read
// copy; at head width 128 this also frees the registers the second copy's
// offsets took).
struct DkdvShape {
  int kb, waves, bm, stages, waves_per_eu;
  bool onecopy;  // the ring holds Q and dO once (row-read stride) instead of twice
};
constexpr DkdvShape bwd_dkdv_shape(int head_dim) {
  return head_dim > 96 ? DkdvShape{1, 4, 128, 2, 1, true} : DkdvShape{1, 8, 64, 4, 2, true};
}
constexpr int kBwdDqWaves = 8;
constexpr int kBwdDqBN = 64;
constexpr int kBwdDqStages = 3;
constexpr int kBwdDqStagesD128 = 2;
constexpr bool kBwdDqOneCopy = true;

// Packed windows (runs of short sequences sharing one tile) launch with
// their own shape: fewer wavefronts per workgroup (smaller tiles) and a
// shallower ring -- for the dK/dV pass also 32-query ring tiles -- so that
// two workgroups share a CU; a window then spans at most that many rows.
constexpr int kWinFwdWaves = 4;
constexpr int kWinFwdStages = 3;
constexpr int kWinDqWaves = 4;
constexpr int kWinDqStages = 2;
constexpr int kWinDkdvWaves = 4;
constexpr int kWinDkdvStages = 3;
constexpr int kWinDkdvBM = 32;
constexpr DkdvShape bwd_dkdv_window_shape(int head_dim) {
  return head_dim > 96 ? bwd_dkdv_shape(head_dim)
                       : DkdvShape{1, kWinDkdvWaves, kWinDkdvBM, kWinDkdvStages, bwd_dkdv_shape(head_dim).waves_per_eu,
                                   false};
}
// Every query and key of a packed window lies inside the window, so at head
// widths up to 96 one workgroup computes dQ of its window as well as dK and
// dV (dS goes through LDS instead of being recomputed by the dQ pass), and
// the dQ pass skips the windows.  This needs the two passes to cut the same
// windows (equal window sizes).
constexpr bool bwd_window_fused(int head_dim) {
  return head_dim <= 96 && kWinDkdvBM == 32 && kWinDkdvWaves == kWinDqWaves;
}

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

int fwd_tile_rows(int head_dim);
int bwd_key_tile_rows(int head_dim);
int bwd_query_tile_rows(int head_dim);
// the most rows a packed window of each pass may span
int fwd_window_rows(int head_dim);
int bwd_key_window_rows(int head_dim);
int bwd_query_window_rows(int head_dim);
hipError_t launch_fwd(const FwdArgs& a);
hipError_t launch_bwd(const BwdArgs& a);

// Fills n bf16 values with a deterministic pseudo-random pattern in
// [-1, 1) (used to give profiling runs realistic, finite inputs).
hipError_t launch_fill_bf16(void* p, int64_t n, uint32_t seed, hipStream_t stream);

}  // namespace dcp
