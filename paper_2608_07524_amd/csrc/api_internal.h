// Host-side helpers of the C ABI layer shared by its translation units:
// device checks, work-list uploads and kernel launches.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <initializer_list>

#include "dcp.h"
#include "work_list.h"

namespace dcp {

// DCP_OK when the current device is a gfx950 (its id in *device when not
// null), else DCP_ERR_HIP with the thread's error message set.
int check_device(int* device = nullptr);

// Enqueues on `stream` the copies of the constant chunks to the head of
// `dst` and of each list to its offsets (plan_upload's segments), from a
// library-owned pinned staging buffer, or straight from pageable host memory
// when `pinned` is false (no allocation on the device or of pinned memory).
int upload_head(std::initializer_list<ListAt> lists, void* dst, hipStream_t stream, bool pinned = true);

int check_fwd_tensors(const void* q, const void* k, const void* v, const void* o, const float* lse);

// Launches the forward over `fwd`, whose units and masks are already on the
// device at ws + units_at / ws + windows_at (ws also holds the constants).
int run_fwd(const dcp_attn_desc* d, const UnitList& fwd, const void* q, const void* k, const void* v, void* o,
            float* lse, char* ws, size_t units_at, size_t windows_at, hipStream_t s);

}  // namespace dcp
