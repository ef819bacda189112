// C ABI of libdcp: device checks, work-list uploads, kernel launches, the
// prepared-batch handle and the per-length cost profiler.  Argument
// validation and the work lists themselves are host code (work_list.cpp).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "attn_common.h"
#include "attn_launch.h"
#include "api_internal.h"
#include "dcp_internal.h"
#include "work_list.h"

namespace dcp {

KernelEvents& kernel_events() {
  thread_local KernelEvents ev;
  return ev;
}

// The kernels are built for gfx950 only; refuse other devices up front.
int check_device(int* device) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "no HIP device: %s", hipGetErrorString(e));
  if (device) *device = dev;
  static std::mutex mu;
  static std::vector<int> ok_devices;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (std::find(ok_devices.begin(), ok_devices.end(), dev) != ok_devices.end()) return DCP_OK;
  }
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(DCP_ERR_HIP, "device %d is %s; libdcp is built for gfx950 only", dev, prop.gcnArchName);
  std::lock_guard<std::mutex> lock(mu);
  ok_devices.push_back(dev);
  return DCP_OK;
}

namespace {

// Pinned host staging for the work-list copies: per device a ring of
// library-owned pinned buffers, each with an event marking when the copy
// out of it has run, so that a buffer is rewritten only after its last copy.
// A copy from pageable memory passes through the runtime's own staging and
// held the host until the stream had drained the work queued before it
// (for a backward call behind another, the whole pass); from pinned memory
// the host only enqueues.  When a list outgrows the ring, every slot moves to
// new buffers of the next power of two (at least 1 MiB) and the old ones are
// kept, never freed: freeing pinned memory waits for the device, and a copy
// may still be reading them.  What is kept stays below the ring's own size.
// (The no-allocation forward keeps the pageable copy: these are allocations.)
constexpr int kStageSlots = 4;
struct StageSlot {
  unsigned char* host = nullptr;
  hipEvent_t done = nullptr;
  bool pending = false;
};
struct StageRing {
  int dev = -1;
  size_t cap = 0;
  unsigned next = 0;
  StageSlot slot[kStageSlots];
  std::vector<void*> retired;
};
std::mutex g_stage_mu;
std::vector<StageRing*> g_rings;  // one per device, kept until the process ends

int grow_ring(StageRing* r, size_t bytes) {
  size_t cap = size_t(1) << 20;
  while (cap < bytes) cap *= 2;
  for (StageSlot& sl : r->slot) {
    void* p = nullptr;
    const hipError_t e = hipHostMalloc(&p, cap, hipHostMallocDefault);
    if (e != hipSuccess) return fail(DCP_ERR_HIP, "pinned staging of %zu bytes: %s", cap, hipGetErrorString(e));
    if (sl.host) r->retired.push_back(sl.host);
    sl.host = static_cast<unsigned char*>(p);
    sl.pending = false;  // the new buffer has no copy in flight
  }
  r->cap = cap;
  return DCP_OK;
}

// One copy per segment, from the host buffer fill_segments wrote.
int copy_segments(const UploadPlan& u, const unsigned char* buf, void* dst, hipStream_t stream) {
  size_t off = 0;
  for (const UploadSegment& g : u.segs) {
    const hipError_t e =
        hipMemcpyAsync(static_cast<char*>(dst) + g.at, buf + off, g.end - g.at, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return fail(DCP_ERR_HIP, "work list upload: %s", hipGetErrorString(e));
    off += g.end - g.at;
  }
  return DCP_OK;
}

int upload_pinned(const UploadPlan& u, void* dst, hipStream_t stream) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lock(g_stage_mu);
  StageRing* ring = nullptr;
  for (StageRing* r : g_rings)
    if (r->dev == dev) ring = r;
  if (!ring) {
    ring = new (std::nothrow) StageRing{};
    if (!ring) return fail(DCP_ERR_INVALID, "out of host memory");
    ring->dev = dev;
    g_rings.push_back(ring);
  }
  int st;
  if (ring->cap < u.bytes && (st = grow_ring(ring, u.bytes))) return st;
  StageSlot& sl = ring->slot[ring->next++ % kStageSlots];
  if (sl.pending && (e = hipEventSynchronize(sl.done)) != hipSuccess)
    return fail(DCP_ERR_HIP, "work list staging: %s", hipGetErrorString(e));
  sl.pending = false;
  if (!sl.done && (e = hipEventCreateWithFlags(&sl.done, hipEventDisableTiming)) != hipSuccess)
    return fail(DCP_ERR_HIP, "staging event: %s", hipGetErrorString(e));
  fill_segments(u, sl.host);
  if ((st = copy_segments(u, sl.host, dst, stream))) return st;
  if ((e = hipEventRecord(sl.done, stream)) != hipSuccess)
    return fail(DCP_ERR_HIP, "work list staging: %s", hipGetErrorString(e));
  sl.pending = true;
  return DCP_OK;
}

}  // namespace

// The constant chunks and the lists as plan_upload's segments, through the
// pinned staging ring unless `pinned` is false (the per-row areas after the
// last list, and the space reserved between segments, are not touched).
int upload_head(std::initializer_list<ListAt> lists, void* dst, hipStream_t stream, bool pinned) {
  UploadPlan u;
  std::vector<unsigned char> img;
  try {
    u = plan_upload(lists.begin(), lists.size());
    if (!pinned) img.resize(u.bytes);
  } catch (const std::bad_alloc&) {
    return fail(DCP_ERR_INVALID, "out of host memory staging the work lists");
  }
  if (pinned) return upload_pinned(u, dst, stream);
  fill_segments(u, img.data());
  return copy_segments(u, img.data(), dst, stream);
}

int check_fwd_tensors(const void* q, const void* k, const void* v, const void* o, const float* lse) {
  int st;
  if ((st = check_tensor(q, "q")) || (st = check_tensor(k, "k")) || (st = check_tensor(v, "v")) ||
      (st = check_tensor(o, "o")))
    return st;
  if (!lse || reinterpret_cast<uintptr_t>(lse) % 4) return fail(DCP_ERR_INVALID, "lse is null or misaligned");
  return DCP_OK;
}

int check_bwd_tensors(const void* dout, const void* o, const float* lse, const void* q, const void* k,
                      const void* v, const void* dq, const void* dk, const void* dv) {
  int st;
  if ((st = check_tensor(dout, "dout")) || (st = check_tensor(o, "o")) || (st = check_tensor(q, "q")) ||
      (st = check_tensor(k, "k")) || (st = check_tensor(v, "v")) || (st = check_tensor(dq, "dq")) ||
      (st = check_tensor(dk, "dk")) || (st = check_tensor(dv, "dv")))
    return st;
  if (!lse || reinterpret_cast<uintptr_t>(lse) % 4) return fail(DCP_ERR_INVALID, "lse is null or misaligned");
  return DCP_OK;
}

// Launches the forward over `fwd` (its units and masks already on the
// device at ws + units_at / windows_at).
int run_fwd(const dcp_attn_desc* d, const UnitList& fwd, const void* q, const void* k, const void* v, void* o,
            float* lse, char* ws, size_t units_at, size_t windows_at, hipStream_t s) {
  FwdArgs a{q, k, v, o, lse, ws, ws + units_at, ws + windows_at, int(fwd.n_tiles),
            int(fwd.units.size() - fwd.n_tiles), d->n_heads, d->head_dim, int(d->total_tokens),
            d->scale, d->causal, s};
  hipError_t e = launch_fwd(a);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "forward launch: %s", hipGetErrorString(e));
  return DCP_OK;
}

int run_bwd(const dcp_attn_desc* d, const UnitList& kl, const UnitList& ql, const void* dout, const void* o,
            const float* lse, const void* q, const void* k, const void* v, void* dq, void* dk, void* dv, char* ws,
            size_t units_at, size_t windows_at, size_t qunits_at, size_t qwindows_at, size_t lse2_at,
            size_t delta_at, hipStream_t s) {
  BwdArgs a{dout, o, lse, q, k, v, dq, dk, dv, reinterpret_cast<float*>(ws + delta_at),
            reinterpret_cast<float*>(ws + lse2_at), ws, ws + units_at, ws + windows_at, int(kl.n_tiles),
            int(kl.units.size() - kl.n_tiles), ws + qunits_at, ws + qwindows_at, int(ql.n_tiles),
            int(ql.units.size() - ql.n_tiles), d->cu_seqlens_host[d->n_seqs], d->n_heads, d->head_dim,
            int(d->total_tokens), d->scale, d->causal, s};
  hipError_t e = launch_bwd(a);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "backward launch: %s", hipGetErrorString(e));
  return DCP_OK;
}

namespace {

// A batch's workspace must be the buffer its lists were uploaded into, on
// the current device, and large enough.
int check_batch_ws(const dcp_batch_s* b, const void* ws, size_t bytes) {
  if (!b) return fail(DCP_ERR_INVALID, "batch is null");
  if (!ws || bytes < b->total)
    return fail(DCP_ERR_WORKSPACE, "batch workspace needs %zu bytes, got %zu", b->total, bytes);
  if (ws != b->uploaded) return fail(DCP_ERR_INVALID, "workspace is not the buffer dcp_batch_upload filled");
  int dev = -1;
  int st = check_device(&dev);
  if (st) return st;
  if (dev != b->device) return fail(DCP_ERR_INVALID, "the batch was uploaded on device %d, current is %d", b->device, dev);
  return DCP_OK;
}

}  // namespace
}  // namespace dcp

using namespace dcp;

extern "C" int dcp_set_kernel_events(void* begin, void* end) {
  clear_error();
  if ((begin == nullptr) != (end == nullptr)) return fail(DCP_ERR_INVALID, "set both events or neither");
  kernel_events().begin = static_cast<hipEvent_t>(begin);
  kernel_events().end = static_cast<hipEvent_t>(end);
  return DCP_OK;
}

extern "C" int dcp_device_info(int32_t* compute_units, int32_t* clock_khz) {
  clear_error();
  if (!compute_units || !clock_khz) return fail(DCP_ERR_INVALID, "outputs are null");
  int dev = -1;
  int st = check_device(&dev);
  if (st) return st;
  int cus = 0, khz = 0;
  hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeClockRate, dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
  *compute_units = cus;
  *clock_khz = khz;
  return DCP_OK;
}

extern "C" int dcp_varlen_attn_fwd_workspace_size(const dcp_attn_desc* desc, size_t* bytes) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if (!bytes) return fail(DCP_ERR_INVALID, "bytes is null");
  *bytes = fwd_layout(desc).total;
  return DCP_OK;
}

extern "C" int dcp_varlen_attn_bwd_workspace_size(const dcp_attn_desc* desc, size_t* bytes) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if (!bytes) return fail(DCP_ERR_INVALID, "bytes is null");
  *bytes = bwd_layout(desc).total;
  return DCP_OK;
}

extern "C" int dcp_varlen_attn_fwd(const dcp_attn_desc* desc, const void* q, const void* k, const void* v, void* o,
                                   float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if ((st = check_fwd_tensors(q, k, v, o, lse))) return st;
  const FwdLayout l = fwd_layout(desc);
  if (!workspace || workspace_bytes < l.total)
    return fail(DCP_ERR_WORKSPACE, "forward workspace needs %zu bytes, got %zu", l.total, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(DCP_ERR_INVALID, "workspace must be 16-byte aligned");
  if ((st = check_device())) return st;
  const UnitList units = build_pass(desc, kPassFwd);
  if (units.units.empty()) return DCP_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = upload_head({{l.units, l.windows, &units}}, workspace, s))) return st;
  return run_fwd(desc, units, q, k, v, o, lse, static_cast<char*>(workspace), l.units, l.windows, s);
}

extern "C" int dcp_varlen_attn_bwd(const dcp_attn_desc* desc, const void* dout, const void* o, const float* lse,
                                   const void* q, const void* k, const void* v, void* dq, void* dk, void* dv,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if ((st = check_bwd_tensors(dout, o, lse, q, k, v, dq, dk, dv))) return st;
  const BwdLayout l = bwd_layout(desc);
  if (!workspace || workspace_bytes < l.total)
    return fail(DCP_ERR_WORKSPACE, "backward workspace needs %zu bytes, got %zu", l.total, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(DCP_ERR_INVALID, "workspace must be 16-byte aligned");
  if ((st = check_device())) return st;
  const UnitList units = build_pass(desc, kPassDkdv);
  if (units.units.empty()) return DCP_OK;
  const UnitList qunits = build_pass(desc, kPassDq);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = upload_head({{l.units, l.windows, &units}, {l.qunits, l.qwindows, &qunits}}, workspace, s))) return st;
  return run_bwd(desc, units, qunits, dout, o, lse, q, k, v, dq, dk, dv, static_cast<char*>(workspace), l.units,
                 l.windows, l.qunits, l.qwindows, l.lse2, l.delta, s);
}

// ---------------------------------------------------------------------------
// Prepared batches.

extern "C" int dcp_batch_create(const dcp_attn_desc* desc, dcp_batch* out) {
  clear_error();
  if (!out) return fail(DCP_ERR_INVALID, "out is null");
  *out = nullptr;
  dcp_batch_s* b = new (std::nothrow) dcp_batch_s();
  if (!b) return fail(DCP_ERR_INVALID, "out of host memory");
  int st;
  try {
    st = batch_init(desc, b);
  } catch (const std::bad_alloc&) {
    st = fail(DCP_ERR_INVALID, "out of host memory building the work lists");
  }
  if (st) {
    delete b;
    return st;
  }
  *out = b;
  return DCP_OK;
}

extern "C" void dcp_batch_destroy(dcp_batch b) { delete b; }

extern "C" int dcp_batch_workspace_size(dcp_batch b, size_t* bytes) {
  clear_error();
  if (!b || !bytes) return fail(DCP_ERR_INVALID, "batch or bytes is null");
  *bytes = b->total;
  return DCP_OK;
}

extern "C" int dcp_batch_upload(dcp_batch b, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  if (!b) return fail(DCP_ERR_INVALID, "batch is null");
  if (!workspace || workspace_bytes < b->total)
    return fail(DCP_ERR_WORKSPACE, "batch workspace needs %zu bytes, got %zu", b->total, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 256) return fail(DCP_ERR_INVALID, "workspace must be 256-byte aligned");
  int dev = -1;
  int st = check_device(&dev);
  if (st) return st;
  st = upload_head({{b->units_at[kPassFwd], b->windows_at[kPassFwd], &b->pass[kPassFwd]},
                    {b->units_at[kPassDkdv], b->windows_at[kPassDkdv], &b->pass[kPassDkdv]},
                    {b->units_at[kPassDq], b->windows_at[kPassDq], &b->pass[kPassDq]}},
                   workspace, static_cast<hipStream_t>(stream));
  if (st) return st;
  b->uploaded = workspace;
  b->device = dev;
  return DCP_OK;
}

extern "C" int dcp_batch_fwd(dcp_batch b, const void* q, const void* k, const void* v, void* o, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  int st = check_batch_ws(b, workspace, workspace_bytes);
  if (st) return st;
  if ((st = check_fwd_tensors(q, k, v, o, lse))) return st;
  const UnitList& f = b->pass[kPassFwd];
  if (f.units.empty()) return DCP_OK;
  return run_fwd(&b->desc, f, q, k, v, o, lse, static_cast<char*>(workspace), b->units_at[kPassFwd],
                 b->windows_at[kPassFwd], static_cast<hipStream_t>(stream));
}

extern "C" int dcp_batch_bwd(dcp_batch b, const void* dout, const void* o, const float* lse, const void* q,
                             const void* k, const void* v, void* dq, void* dk, void* dv, void* workspace,
                             size_t workspace_bytes, void* stream) {
  clear_error();
  int st = check_batch_ws(b, workspace, workspace_bytes);
  if (st) return st;
  if ((st = check_bwd_tensors(dout, o, lse, q, k, v, dq, dk, dv))) return st;
  if (b->pass[kPassDkdv].units.empty()) return DCP_OK;
  return run_bwd(&b->desc, b->pass[kPassDkdv], b->pass[kPassDq], dout, o, lse, q, k, v, dq, dk, dv,
                 static_cast<char*>(workspace), b->units_at[kPassDkdv], b->windows_at[kPassDkdv],
                 b->units_at[kPassDq], b->windows_at[kPassDq], b->lse2_at, b->delta_at,
                 static_cast<hipStream_t>(stream));
}

extern "C" int dcp_work_list(const dcp_attn_desc* desc, int32_t pass, int32_t* units, size_t cap, size_t* n_units,
                             size_t* n_tiles, uint64_t* window_starts, size_t cap_windows, size_t* n_windows) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if (!n_units || !n_tiles || !n_windows) return fail(DCP_ERR_INVALID, "count outputs are null");
  if (pass < kPassFwd || pass > kPassDq) return fail(DCP_ERR_INVALID, "pass must be 0 (forward), 1 (dK/dV) or 2 (dQ)");
  const UnitList l = build_pass(desc, pass);
  const size_t nw = l.window_starts.size() / kWindowWords;
  if (units && cap < l.units.size()) return fail(DCP_ERR_INVALID, "units holds %zu, need %zu", cap, l.units.size());
  if (window_starts && cap_windows < nw) return fail(DCP_ERR_INVALID, "window_starts holds %zu, need %zu", cap_windows, nw);
  *n_units = l.units.size();
  *n_tiles = l.n_tiles;
  *n_windows = nw;
  if (units)
    for (size_t i = 0; i < l.units.size(); ++i) {
      const WorkUnit& u = l.units[i];
      int32_t* o = units + 5 * i;
      o[0] = u.row0;
      o[1] = u.seq0;
      o[2] = u.seqlen;
      o[3] = u.rows;
      o[4] = u.head;
    }
  if (window_starts && nw) std::memcpy(window_starts, l.window_starts.data(), l.window_starts.size() * sizeof(uint64_t));
  return DCP_OK;
}

// ---------------------------------------------------------------------------
// Per-length cost profile.

namespace {

int validate_profile_opts(const dcp_profile_opts* o) {
  if (!o) return fail(DCP_ERR_INVALID, "profile opts are null");
  if (o->n_heads < 1) return fail(DCP_ERR_INVALID, "n_heads must be >= 1");
  if (o->head_dim != 64 && o->head_dim != 72 && o->head_dim != 128)
    return fail(DCP_ERR_UNSUPPORTED, "head_dim %d is not supported (64, 72, 128)", o->head_dim);
  if (o->causal != 0 && o->causal != 1) return fail(DCP_ERR_INVALID, "causal must be 0 or 1");
  if (!std::isfinite(o->scale)) return fail(DCP_ERR_INVALID, "scale must be finite");
  if (o->warmup < 0 || o->reps < 1) return fail(DCP_ERR_INVALID, "need warmup >= 0 and reps >= 1");
  if (o->lin_f_ps_per_token < 0 || o->lin_b_ps_per_token < 0 || o->act_bytes_per_token < 0 ||
      o->inp_bytes_per_token < 0)
    return fail(DCP_ERR_INVALID, "per-token terms must be non-negative");
  return DCP_OK;
}

struct ProfLayout {
  size_t tensor;  // bytes of one [max_len, H, D] bf16 tensor
  size_t lse;
  size_t ws_off;
  size_t ws_bytes;
  size_t total;
};

ProfLayout prof_layout(int64_t max_len, const dcp_profile_opts* o) {
  ProfLayout l;
  l.tensor = align_up(size_t(max_len) * size_t(o->n_heads) * size_t(o->head_dim) * 2);
  l.lse = align_up(size_t(max_len) * size_t(o->n_heads) * 4);
  // a prepared batch of the longest length: its lists and scratch bound
  // every shorter length's
  int32_t cu[2] = {0, int32_t(max_len)};
  dcp_attn_desc d{1, cu, max_len, o->n_heads, o->head_dim, 1.f, o->causal};
  dcp_batch_s b;
  l.ws_bytes = batch_init(&d, &b) == DCP_OK ? b.total : 0;
  l.ws_off = 8 * l.tensor + l.lse;
  l.total = l.ws_off + l.ws_bytes;
  return l;
}

}  // namespace

extern "C" int dcp_profile_workspace_size(int64_t max_len, const dcp_profile_opts* opts, size_t* bytes) {
  clear_error();
  int st = validate_profile_opts(opts);
  if (st) return st;
  if (max_len < 1 || max_len >= (int64_t(1) << 31)) return fail(DCP_ERR_INVALID, "max_len must be in [1, 2^31)");
  if (!bytes) return fail(DCP_ERR_INVALID, "bytes is null");
  *bytes = prof_layout(max_len, opts).total;
  return DCP_OK;
}

extern "C" int dcp_profile_cost(const int64_t* lengths, int32_t n, const dcp_profile_opts* opts, void* workspace,
                                size_t workspace_bytes, void* stream, dcp_cost_row* out_rows) {
  clear_error();
  int st = validate_profile_opts(opts);
  if (st) return st;
  if (n < 1 || !lengths || !out_rows) return fail(DCP_ERR_INVALID, "need n >= 1 lengths and an output array");
  int64_t max_len = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (lengths[i] < 1 || lengths[i] >= (int64_t(1) << 31))
      return fail(DCP_ERR_INVALID, "length %lld out of range", static_cast<long long>(lengths[i]));
    max_len = std::max(max_len, lengths[i]);
  }
  const ProfLayout l = prof_layout(max_len, opts);
  if (!workspace || workspace_bytes < l.total)
    return fail(DCP_ERR_WORKSPACE, "profile workspace needs %zu bytes for length %lld, got %zu", l.total,
                static_cast<long long>(max_len), workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 256) return fail(DCP_ERR_INVALID, "workspace must be 256-byte aligned");
  if ((st = check_device())) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  void* t[8];
  for (int i = 0; i < 8; ++i) t[i] = ws + size_t(i) * l.tensor;
  float* lse = reinterpret_cast<float*>(ws + 8 * l.tensor);
  void* aws = ws + l.ws_off;
  const int64_t elems = max_len * int64_t(opts->n_heads) * opts->head_dim;
  for (int i = 0; i < 5; ++i) {  // q, k, v, o, dO
    hipError_t e = launch_fill_bf16(t[i], elems, 0x1234567u + 977u * uint32_t(i), s);
    if (e != hipSuccess) return fail(DCP_ERR_HIP, "fill: %s", hipGetErrorString(e));
  }
  const float scale = opts->scale > 0.f ? opts->scale : 1.f / std::sqrt(float(opts->head_dim));
  // Per length: the work lists are built and uploaded once, before any
  // timing; then every warm-up and timed run is enqueued back to back (the
  // host only launches, so it stays ahead of the device) with events around
  // the forward and the backward of each timed run, and one synchronisation
  // at the end.  The times are device time between the events.
  const int32_t reps = opts->reps;
  std::vector<hipEvent_t> ev(size_t(3 * reps), nullptr);
  for (auto& e : ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      for (auto& x : ev)
        if (x) (void)hipEventDestroy(x);
      return fail(DCP_ERR_HIP, "hipEventCreate failed");
    }
  }
  std::vector<dcp_cost_row> rows(static_cast<size_t>(n));
  int result = DCP_OK;
  for (int32_t i = 0; i < n && result == DCP_OK; ++i) {
    const int64_t len = lengths[i];
    int32_t cu[2] = {0, int32_t(len)};
    dcp_attn_desc d{1, cu, len, opts->n_heads, opts->head_dim, scale, opts->causal};
    dcp_batch_s b;
    if ((result = batch_init(&d, &b))) break;
    if (b.total > l.ws_bytes) {
      result = fail(DCP_ERR_WORKSPACE, "length %lld needs %zu workspace bytes", static_cast<long long>(len), b.total);
      break;
    }
    if ((result = dcp_batch_upload(&b, aws, l.ws_bytes, stream))) break;
    for (int32_t r = 0; r < opts->warmup + reps && result == DCP_OK; ++r) {
      const int32_t k = r - opts->warmup;  // timed run index (< 0: warm-up)
      if (k >= 0) (void)hipEventRecord(ev[size_t(3 * k)], s);
      result = dcp_batch_fwd(&b, t[0], t[1], t[2], t[3], lse, aws, l.ws_bytes, stream);
      if (result) break;
      if (k >= 0) (void)hipEventRecord(ev[size_t(3 * k + 1)], s);
      result = dcp_batch_bwd(&b, t[4], t[3], lse, t[0], t[1], t[2], t[5], t[6], t[7], aws, l.ws_bytes, stream);
      if (result) break;
      if (k >= 0) (void)hipEventRecord(ev[size_t(3 * k + 2)], s);
    }
    if (result) break;
    if (hipEventSynchronize(ev[size_t(3 * reps - 1)]) != hipSuccess) {
      result = fail(DCP_ERR_HIP, "profile run failed: %s", hipGetErrorString(hipGetLastError()));
      break;
    }
    std::vector<float> tf, tb;
    for (int32_t k = 0; k < reps; ++k) {
      float a = 0.f, c = 0.f;
      (void)hipEventElapsedTime(&a, ev[size_t(3 * k)], ev[size_t(3 * k + 1)]);
      (void)hipEventElapsedTime(&c, ev[size_t(3 * k + 1)], ev[size_t(3 * k + 2)]);
      tf.push_back(a);
      tb.push_back(c);
    }
    std::sort(tf.begin(), tf.end());
    std::sort(tb.begin(), tb.end());
    const double mf = tf[tf.size() / 2], mb = tb[tb.size() / 2];
    dcp_cost_row& row = rows[size_t(i)];
    row.seq_len = len;
    row.t_f_ns = int64_t(std::llround(mf * 1e6)) + opts->lin_f_ps_per_token * len / 1000;
    row.t_b_ns = int64_t(std::llround(mb * 1e6)) + opts->lin_b_ps_per_token * len / 1000;
    row.m_bytes = len * opts->act_bytes_per_token;
    row.m_inp_bytes = len * opts->inp_bytes_per_token;
  }
  for (auto& e : ev) (void)hipEventDestroy(e);
  if (result) return result;
  std::memcpy(out_rows, rows.data(), sizeof(dcp_cost_row) * size_t(n));
  return DCP_OK;
}
