// Host-side work lists of the attention kernels: argument validation, the
// tile lists of each kernel pass built from cu_seqlens, and the byte layouts
// of the workspaces that carry them to the device.  Plain C++ (no HIP): the
// lists are built on the host and copied to the device by the ABI layer.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "dcp.h"
#include "tile_shapes.h"

namespace dcp {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// DCP_OK, or the status (with the thread's error message set) for a bad
// descriptor: cu_seqlens, sizes, head width, scale, causal flag.
int validate_desc(const dcp_attn_desc* d);
// A non-null, 16-byte aligned device tensor pointer.
int check_tensor(const void* p, const char* name);

struct UnitList {
  std::vector<WorkUnit> units;  // n_tiles sequence tiles, then the packed windows (8 per-die lists each)
  size_t n_tiles = 0;
  std::vector<uint64_t> window_starts;  // kWindowWords per packed window
};

// The kernel passes and their lists.
enum : int32_t { kPassFwd = 0, kPassDkdv = 1, kPassDq = 2 };
UnitList build_units(const dcp_attn_desc* d, int tile, int window_tile, bool keys_major);
UnitList build_pass(const dcp_attn_desc* d, int32_t pass);

// Bytes reserved for one pass's list and for its window masks (upper
// bounds, padding included, for workspaces sized before the list exists).
size_t list_bytes(const dcp_attn_desc* d, int tile);
size_t window_bytes(const dcp_attn_desc* d, int tile);

// The 16-byte constant chunks every attention workspace starts with
// (bf16 [0 x 8], bf16 [1, 0 x 7], fp32 +inf).
void const_head(unsigned char (&head)[kConstBytes]);

// Forward workspace: constant chunks | tile list | its window masks.
struct FwdLayout {
  size_t units, windows, total;
};
FwdLayout fwd_layout(const dcp_attn_desc* d);

// Backward workspace: constant chunks | key-tile list | its window masks |
// query-tile list | its window masks | LSE*log2e [H, T] | -Delta [H, T].
struct BwdLayout {
  size_t units, windows, qunits, qwindows, lse2, delta, total;
};
BwdLayout bwd_layout(const dcp_attn_desc* d);

// One work list with its window masks, to be copied to byte offsets
// units_at / windows_at of a device buffer.
struct ListAt {
  size_t units_at, windows_at;
  const UnitList* list;
};
// What an upload writes: the constant chunks at offset 0 and each list and
// its window masks at their offsets.  A per-call workspace reserves room for
// the longest possible list ahead of the next one, so these parts can lie
// megabytes apart: parts at most kMergeGap apart form one segment (the bytes
// between them zeroed), the others segments of their own, which a host
// buffer holds back to back; the space between segments is neither filled
// nor copied.
constexpr size_t kMergeGap = size_t(16) << 10;
struct UploadPart {
  size_t at, bytes;
  const void* src;  // null: the constant chunks
};
struct UploadSegment {
  size_t at, end;  // device byte range
};
struct UploadPlan {
  std::vector<UploadPart> parts;  // by offset
  std::vector<UploadSegment> segs;
  size_t bytes = 0;  // host bytes: the segments back to back
};
UploadPlan plan_upload(const ListAt* lists, size_t n_lists);
// Writes the segments back to back into `buf` (plan.bytes bytes).
void fill_segments(const UploadPlan& plan, unsigned char* buf);

}  // namespace dcp

// A prepared batch (dcp_batch in dcp.h): a copy of the descriptor and of
// cu_seqlens, the lists of all three passes, and the byte layout of the
// device buffer they are uploaded into:
//   constant chunks | forward list | its masks | dK/dV list | its masks |
//   dQ list | its masks | LSE*log2e [H, T] | -Delta [H, T]
// (each part 256-byte aligned, the lists at their exact sizes).
struct dcp_batch_s {
  dcp_attn_desc desc{};
  std::vector<int32_t> cu;
  dcp::UnitList pass[3];
  size_t units_at[3] = {0, 0, 0}, windows_at[3] = {0, 0, 0};
  size_t lse2_at = 0, delta_at = 0, total = 0;
  // the buffer last uploaded into and its device (-1: none yet)
  const void* uploaded = nullptr;
  int device = -1;
};

namespace dcp {
// Validates `desc` and fills `b` (host work only).
int batch_init(const dcp_attn_desc* desc, dcp_batch_s* b);
}  // namespace dcp
