// The attention forward for callers that cannot allocate device memory:
// its scratch (the constant chunks, the work list and the window masks)
// lives in a fixed-size device array of this library instead of a
// caller-provided workspace.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "api_internal.h"
#include "dcp_internal.h"
#include "work_list.h"

namespace dcp {
namespace {

constexpr size_t kScratchBytes = size_t(8) << 20;  // the limit stated in dcp.h

// One copy per device, held until the process ends.  Host code never uses
// this name as an address: it takes each device's address from
// hipGetSymbolAddress (scratch_ptr below).
static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
std::vector<std::pair<int, void*>> g_ptr;  // (device, address of its scratch)

// Address of `scratch` on the current device `dev`, looked up once per
// device (with that device current) and kept.
int scratch_ptr(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  for (const auto& e : g_ptr)
    if (e.first == dev) {
      *out = e.second;
      return DCP_OK;
    }
  void* p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr)
    return fail(DCP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
  g_ptr.emplace_back(dev, p);
  *out = p;
  return DCP_OK;
}

}  // namespace
}  // namespace dcp

using namespace dcp;

extern "C" int dcp_varlen_attn_fwd_noalloc(const dcp_attn_desc* desc, const void* q, const void* k, const void* v,
                                           void* o, float* lse, void* stream) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if ((st = check_fwd_tensors(q, k, v, o, lse))) return st;
  UnitList units;
  try {
    units = build_pass(desc, kPassFwd);
  } catch (const std::bad_alloc&) {
    return fail(DCP_ERR_INVALID, "out of host memory building the work list");
  }
  // constants | units | window masks, each part 256-byte aligned
  const size_t units_at = kConstBytes;
  const size_t windows_at = units_at + align_up(std::max<size_t>(1, units.units.size()) * sizeof(WorkUnit));
  const size_t need = windows_at + align_up(std::max<size_t>(1, units.window_starts.size()) * sizeof(uint64_t));
  if (need > kScratchBytes)
    return fail(DCP_ERR_WORKSPACE, "the forward's work list needs %zu bytes of scratch; the fixed scratch holds %zu",
                need, kScratchBytes);
  int dev = -1;
  if ((st = check_device(&dev))) return st;
  if (units.units.empty()) return DCP_OK;
  void* ws = nullptr;
  if ((st = scratch_ptr(dev, &ws))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = upload_head({{units_at, windows_at, &units}}, ws, s, /*pinned=*/false))) return st;
  return run_fwd(desc, units, q, k, v, o, lse, static_cast<char*>(ws), units_at, windows_at, s);
}
