// Tile shapes and the work-unit record shared by the host code that builds
// work lists and the HIP kernels that consume them.  Plain C++ (no HIP
// headers), so the host-side list builder also compiles on its own.
#pragma once

#include <stdint.h>

namespace dcp {

// One tile of work: rows [row0, row0 + rows) of the packed tensor for head
// `head`, all in the sequence that occupies rows [seq0, seq0 + seqlen).
// rows == 0 marks padding (the workgroup exits at once).
// A negative seqlen marks a packed window instead: consecutive sequences,
// each shorter than a tile, sharing one tile of `rows` rows that starts at
// row0 == seq0.  Row i of the window attends only to rows of its own
// sequence; -seqlen - 1 indexes the window's mask of sequence starts (four
// 64-bit words, bit x set where a sequence starts at window offset x).
struct WorkUnit {
  int32_t row0;
  int32_t seq0;
  int32_t seqlen;
  uint16_t rows;  // at most one tile (256)
  uint16_t head;  // head counts are limited to 65535 by the C ABI
};
static_assert(sizeof(WorkUnit) == 16, "16 bytes per tile");
constexpr int kWindowWords = 4;  // 64-bit words per window mask: windows hold at most 256 rows

constexpr int kNumXcd = 8;  // MI355X: 8 accelerator dies, each with its own L2

// Offsets (bf16 elements) of the 16-byte constant chunks every attention
// workspace starts with.
constexpr int kConstZero = 0;   // [0, 0, 0, 0, 0, 0, 0, 0]
constexpr int kConstOnes = 8;   // [1, 0, 0, 0, 0, 0, 0, 0]
constexpr int kConstInf = 16;   // fp32 +inf (a query past its sequence end)
constexpr int kConstBytes = 256;

// Query rows per forward workgroup: kFwdWaves wavefronts x 32.
constexpr int kFwdWaves = 8;
// Backward, dK/dV pass: `waves` wavefronts per workgroup, each owning
// 32*kb keys whose K, V fragments and dK, dV accumulators stay resident,
// stepping over `bm` queries at a time through a `stages`-deep LDS ring;
// waves_per_eu is the occupancy the register allocation must allow.
// Head widths up to 72 run two wavefronts of 32 keys per SIMD, with Q and
// dO held once per ring stage (the transposing reads of dV and dK use the
// row-read copy, at the cost of some bank conflicts), which leaves LDS for
// a four-stage ring of 64-query tiles.  At head width 128, K and V
// fragments plus the dK, dV accumulators would need more than the 256
// registers two wavefronts per SIMD can each have; V is therefore read from
// an LDS copy of the tile's 256 V rows (68 KB), which leaves K, the
// accumulators and one 16-column step of operands in registers (249-256),
// and the ring holds Q and dO once in two stages of 64-query tiles (76 KB).
// dQ pass: kBwdDqWaves wavefronts of 32 queries, kBwdDqBN keys per step,
// K held once per ring stage (its transposing reads share the row-read
// copy; at head width 128 this also frees the registers the second copy's
// offsets took).
struct DkdvShape {
  int kb, waves, bm, stages, waves_per_eu;
  bool onecopy;  // the ring holds Q and dO once (row-read stride) instead of twice
  bool vlds;     // V fragments read from an LDS copy of the tile's V rows instead of held in registers
};
constexpr DkdvShape bwd_dkdv_shape(int head_dim) {
  return head_dim > 96 ? DkdvShape{1, 8, 64, 2, 2, true, true} : DkdvShape{1, 8, 64, 4, 2, true, false};
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
                                   false, false};
}
// Every query and key of a packed window lies inside the window, so at head
// widths up to 96 one workgroup computes dQ of its window as well as dK and
// dV (dS goes through LDS instead of being recomputed by the dQ pass), and
// the dQ pass skips the windows.  This needs the two passes to cut the same
// windows (equal window sizes).
constexpr bool bwd_window_fused(int head_dim) {
  return head_dim <= 96 && kWinDkdvBM == 32 && kWinDkdvWaves == kWinDqWaves;
}

// Rows per tile of each pass, and the most rows a packed window of each pass
// may span.
constexpr int fwd_tile_rows(int) { return kFwdWaves * 32; }
constexpr int fwd_window_rows(int) { return kWinFwdWaves * 32; }
constexpr int bwd_key_tile_rows(int head_dim) {
  return 32 * bwd_dkdv_shape(head_dim).kb * bwd_dkdv_shape(head_dim).waves;
}
constexpr int bwd_query_tile_rows(int) { return 32 * kBwdDqWaves; }
constexpr int bwd_key_window_rows(int head_dim) {
  return 32 * bwd_dkdv_window_shape(head_dim).kb * bwd_dkdv_window_shape(head_dim).waves;
}
constexpr int bwd_query_window_rows(int) { return 32 * kWinDqWaves; }

}  // namespace dcp
