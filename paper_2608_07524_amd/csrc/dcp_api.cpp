// C ABI of libdcp: argument validation, work lists, workspace layout,
// kernel launches and the per-length cost profiler.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <limits>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "attn_common.h"
#include "attn_launch.h"
#include "dcp_internal.h"

namespace dcp {

namespace {
thread_local std::string g_last_error;
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

KernelEvents& kernel_events() {
  thread_local KernelEvents ev;
  return ev;
}

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// The kernels are built for gfx950 only; refuse other devices up front.
int check_device() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "no HIP device: %s", hipGetErrorString(e));
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

int validate_desc(const dcp_attn_desc* d) {
  if (!d) return fail(DCP_ERR_INVALID, "desc is null");
  if (d->n_seqs < 1) return fail(DCP_ERR_INVALID, "n_seqs must be >= 1");
  if (!d->cu_seqlens_host) return fail(DCP_ERR_INVALID, "cu_seqlens_host is null");
  if (d->total_tokens < 0 || d->total_tokens >= (int64_t(1) << 31))
    return fail(DCP_ERR_INVALID, "total_tokens must be in [0, 2^31)");
  if (d->n_heads < 1 || d->n_heads > 65535) return fail(DCP_ERR_INVALID, "n_heads must be in [1, 65535]");
  if (d->head_dim != 64 && d->head_dim != 72 && d->head_dim != 128)
    return fail(DCP_ERR_UNSUPPORTED, "head_dim %d is not supported (64, 72, 128)", d->head_dim);
  if (!(std::isfinite(d->scale) && d->scale > 0.f)) return fail(DCP_ERR_INVALID, "scale must be finite and > 0");
  if (d->causal != 0 && d->causal != 1) return fail(DCP_ERR_INVALID, "causal must be 0 or 1");
  const int32_t* cu = d->cu_seqlens_host;
  if (cu[0] != 0) return fail(DCP_ERR_INVALID, "cu_seqlens[0] must be 0");
  for (int32_t b = 0; b < d->n_seqs; ++b)
    if (cu[b + 1] < cu[b]) return fail(DCP_ERR_INVALID, "cu_seqlens must be non-decreasing (index %d)", b + 1);
  if (cu[d->n_seqs] > d->total_tokens)
    return fail(DCP_ERR_INVALID, "cu_seqlens[n] = %d exceeds total_tokens", cu[d->n_seqs]);
  const int64_t elems = d->total_tokens * int64_t(d->n_heads) * d->head_dim;
  if (elems / d->n_heads / d->head_dim != d->total_tokens) return fail(DCP_ERR_INVALID, "tensor size overflows");
  return DCP_OK;
}

int check_tensor(const void* p, const char* name) {
  if (!p) return fail(DCP_ERR_INVALID, "%s is null", name);
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0) return fail(DCP_ERR_INVALID, "%s must be 16-byte aligned", name);
  return DCP_OK;
}

// Tiles of `tile` rows per (sequence, head), never straddling two
// sequences, laid out as 8 per-die lists (see unit_for_block).  Runs of
// consecutive sequences shorter than `window_tile` (<= tile) share one
// tile as a packed window of at most `window_tile` rows (each row still
// attends only within its own sequence), so thousands of short sequences do
// not each occupy a mostly idle workgroup.  Work of a tile: the keys it visits (forward, dQ
// pass) or the queries visiting it (dK/dV pass); a window's is its row
// count.  The (sequence, chunk) and window groups -- long sequences split
// into chunks when a few of them would otherwise leave dies idle -- are
// assigned to the least-loaded die, longest first; each die's list keeps a
// chunk's tiles together (they share K/V or Q/dO in that die's L2) and is
// padded with empty tiles to the longest list.
size_t tiles_per_head(const dcp_attn_desc* d, int tile) {
  size_t n = 0;
  for (int32_t b = 0; b < d->n_seqs; ++b)
    n += size_t((d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b] + tile - 1) / tile);
  return n;
}

struct UnitList {
  std::vector<WorkUnit> units;  // n_tiles sequence tiles, then the packed windows (8 per-die lists each)
  size_t n_tiles = 0;
  std::vector<uint64_t> window_starts;  // kWindowWords per packed window
};

UnitList build_units(const dcp_attn_desc* d, int tile, int window_tile, bool keys_major) {
  const int32_t* cu = d->cu_seqlens_host;
  const int32_t H = d->n_heads;
  const int32_t n = d->n_seqs;
  UnitList out;
  const size_t total = tiles_per_head(d, tile) * size_t(H);
  if (total == 0) return out;
  const size_t cap = std::max<size_t>(4, (total + 8 * kNumXcd - 1) / (8 * kNumXcd));
  // A chunk's work does not depend on its head, so the groups are ordered
  // (longest first) and each expands into its H chunks; thousands of short
  // sequences then cost a sort of the groups only.
  struct Group {
    int64_t work;
    int32_t b, t_begin, t_end;
    int32_t window;  // >= 0: packed window number (b: its first sequence, t_end: its rows)
  };
  std::vector<Group> groups;
  auto tile_work = [&](int32_t len, int32_t t0, int32_t rows) -> int64_t {
    if (!d->causal) return len;
    return keys_major ? int64_t(len) - t0 : int64_t(t0) + rows;
  };
  auto add_sequence = [&](int32_t b) {
    const int32_t len = cu[b + 1] - cu[b];
    const int32_t nt = (len + tile - 1) / tile;
    for (int32_t c0 = 0; c0 < nt; c0 += int32_t(cap)) {
      Group g{0, b, c0, std::min<int32_t>(nt, c0 + int32_t(cap)), -1};
      for (int32_t t = g.t_begin; t < g.t_end; ++t) g.work += tile_work(len, t * tile, std::min(tile, len - t * tile));
      groups.push_back(g);
    }
  };
  for (int32_t b = 0; b < n;) {
    if (cu[b + 1] - cu[b] >= window_tile) {
      add_sequence(b++);
      continue;
    }
    // the run of short sequences from b that fits one window
    int32_t e = b, nonempty = 0, last = b;
    while (e < n && cu[e + 1] - cu[e] < window_tile && cu[e + 1] - cu[b] <= window_tile) {
      if (cu[e + 1] > cu[e]) {
        ++nonempty;
        last = e;
      }
      ++e;
    }
    if (nonempty == 1) {
      add_sequence(last);
    } else if (nonempty > 1) {
      const int32_t w = int32_t(out.window_starts.size() / kWindowWords);
      out.window_starts.resize(out.window_starts.size() + kWindowWords, 0);
      uint64_t* m = &out.window_starts[size_t(w) * kWindowWords];
      const int32_t rows = cu[e] - cu[b];
      for (int32_t i = b; i < e; ++i) {
        const int32_t x = cu[i] - cu[b];
        if (x < rows) m[x / 64] |= uint64_t(1) << (x % 64);
      }
      groups.push_back(Group{rows, b, 0, rows, w});
    }
    b = e;
  }
  std::stable_sort(groups.begin(), groups.end(), [](const Group& x, const Group& y) { return x.work > y.work; });
  // within a chunk, the tile with the most work first (causal: the last
  // query tiles of the forward, the first key tiles of the dK/dV pass)
  const bool reverse = d->causal && !keys_major;
  // sequence tiles and packed windows run as separate launches: each is
  // balanced over the dies on its own
  for (int windows = 0; windows < 2; ++windows) {
    std::vector<std::vector<WorkUnit>> lists(kNumXcd);
    for (auto& l : lists) l.reserve(total / kNumXcd + size_t(cap) + 1);
    int64_t load[kNumXcd] = {0};
    for (const Group& g : groups) {
      if ((g.window >= 0) != (windows == 1)) continue;
      const int32_t s0 = cu[g.b], len = cu[g.b + 1] - cu[g.b];
      for (int32_t h = 0; h < H; ++h) {
        // the least-loaded die takes the chunk
        int x = 0;
        for (int i = 1; i < kNumXcd; ++i)
          if (load[i] < load[x]) x = i;
        load[x] += g.work;
        std::vector<WorkUnit>& l = lists[size_t(x)];
        if (g.window >= 0) {
          WorkUnit u{};
          u.row0 = s0;
          u.seq0 = s0;
          u.seqlen = -g.window - 1;
          u.rows = uint16_t(g.t_end);
          u.head = uint16_t(h);
          l.push_back(u);
          continue;
        }
        for (int32_t i = g.t_begin; i < g.t_end; ++i) {
          const int32_t t = reverse ? g.t_end - 1 - (i - g.t_begin) : i;
          WorkUnit u{};
          u.row0 = s0 + t * tile;
          u.rows = uint16_t(std::min(tile, len - t * tile));
          u.seq0 = s0;
          u.seqlen = len;
          u.head = uint16_t(h);
          l.push_back(u);
        }
      }
    }
    size_t per = 0;
    for (const auto& l : lists) per = std::max(per, l.size());
    const size_t at = out.units.size();
    out.units.resize(at + per * kNumXcd, WorkUnit{});
    for (int x = 0; x < kNumXcd; ++x)
      std::copy(lists[size_t(x)].begin(), lists[size_t(x)].end(), out.units.begin() + ptrdiff_t(at + size_t(x) * per));
    if (windows == 0) out.n_tiles = out.units.size();
  }
  return out;
}

// Upper bound on build_units' length (padding included) for workspace
// sizing: no die list is longer than the total tile count.
size_t count_units(const dcp_attn_desc* d, int tile) {
  return tiles_per_head(d, tile) * size_t(d->n_heads) * kNumXcd;
}

// Bytes reserved for one work list and, after it, its window masks (there
// are fewer windows than tiles of one head).
size_t list_bytes(const dcp_attn_desc* d, int tile) {
  return align_up(sizeof(WorkUnit) * std::max<size_t>(1, count_units(d, tile)));
}
size_t window_bytes(const dcp_attn_desc* d, int tile) {
  return align_up(sizeof(uint64_t) * kWindowWords * std::max<size_t>(1, tiles_per_head(d, tile)));
}

// Backward workspace: constant chunks | key-tile list | its window masks |
// query-tile list | its window masks | LSE*log2e [H, T] | Delta [H, T].
struct BwdLayout {
  size_t units, windows, qunits, qwindows, lse2, delta, total;
};
BwdLayout bwd_layout(const dcp_attn_desc* d) {
  const size_t per_row = align_up(size_t(4) * size_t(d->n_heads) * size_t(d->total_tokens));
  const int kt = bwd_key_tile_rows(d->head_dim), qt = bwd_query_tile_rows(d->head_dim);
  BwdLayout l;
  l.units = kConstBytes;
  l.windows = l.units + list_bytes(d, kt);
  l.qunits = l.windows + window_bytes(d, kt);
  l.qwindows = l.qunits + list_bytes(d, qt);
  l.lse2 = l.qwindows + window_bytes(d, qt);
  l.delta = l.lse2 + per_row;
  l.total = l.delta + per_row;
  return l;
}

// The constant block at the head of a workspace -- 16-byte chunks the
// kernels' direct-to-LDS copies read for pad columns ([0 x 8] and
// [1, 0 x 7] in bf16) and for rows past a sequence end (fp32 +inf) --
// and each work list with its window masks, copied to their byte offsets
// in the workspace (one copy per array: the space reserved between them
// is not touched).
struct ListAt {
  size_t units_at, windows_at;
  const UnitList* list;
};
int upload_head(std::initializer_list<ListAt> lists, void* dst, hipStream_t stream) {
  unsigned char head[kConstBytes] = {};
  const uint16_t one = 0x3F80;  // bf16 1.0
  std::memcpy(head + kConstOnes * 2, &one, sizeof one);
  const float inf = std::numeric_limits<float>::infinity();
  std::memcpy(head + kConstInf * 2, &inf, sizeof inf);
  unsigned char* base = static_cast<unsigned char*>(dst);
  hipError_t e = hipMemcpyAsync(dst, head, sizeof head, hipMemcpyHostToDevice, stream);
  for (const ListAt& l : lists) {
    const UnitList& u = *l.list;
    if (e == hipSuccess && !u.units.empty())
      e = hipMemcpyAsync(base + l.units_at, u.units.data(), u.units.size() * sizeof(WorkUnit), hipMemcpyHostToDevice,
                         stream);
    if (e == hipSuccess && !u.window_starts.empty())
      e = hipMemcpyAsync(base + l.windows_at, u.window_starts.data(), u.window_starts.size() * sizeof(uint64_t),
                         hipMemcpyHostToDevice, stream);
  }
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "work list upload: %s", hipGetErrorString(e));
  return DCP_OK;
}

// Forward workspace: constant chunks | tile list | its window masks.
size_t fwd_windows_at(const dcp_attn_desc* d) { return kConstBytes + list_bytes(d, fwd_tile_rows(d->head_dim)); }
size_t fwd_workspace_bytes(const dcp_attn_desc* d) {
  return fwd_windows_at(d) + window_bytes(d, fwd_tile_rows(d->head_dim));
}

}  // namespace
}  // namespace dcp

using namespace dcp;

extern "C" const char* dcp_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* dcp_version(void) { return "dcp-mi355x 0.1 (gfx950)"; }

extern "C" int dcp_set_kernel_events(void* begin, void* end) {
  clear_error();
  if ((begin == nullptr) != (end == nullptr)) return fail(DCP_ERR_INVALID, "set both events or neither");
  kernel_events().begin = static_cast<hipEvent_t>(begin);
  kernel_events().end = static_cast<hipEvent_t>(end);
  return DCP_OK;
}

extern "C" int dcp_varlen_attn_fwd_workspace_size(const dcp_attn_desc* desc, size_t* bytes) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if (!bytes) return fail(DCP_ERR_INVALID, "bytes is null");
  *bytes = fwd_workspace_bytes(desc);
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
  if ((st = check_tensor(q, "q")) || (st = check_tensor(k, "k")) || (st = check_tensor(v, "v")) ||
      (st = check_tensor(o, "o")))
    return st;
  if (!lse || reinterpret_cast<uintptr_t>(lse) % 4) return fail(DCP_ERR_INVALID, "lse is null or misaligned");
  const int tile = fwd_tile_rows(desc->head_dim);
  const size_t need = fwd_workspace_bytes(desc);
  if (!workspace || workspace_bytes < need)
    return fail(DCP_ERR_WORKSPACE, "forward workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(DCP_ERR_INVALID, "workspace must be 16-byte aligned");
  if ((st = check_device())) return st;
  const UnitList units = build_units(desc, tile, fwd_window_rows(desc->head_dim), false);
  if (units.units.empty()) return DCP_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t windows_at = fwd_windows_at(desc);
  if ((st = upload_head({{kConstBytes, windows_at, &units}}, workspace, s))) return st;
  char* ws = static_cast<char*>(workspace);
  FwdArgs a{q, k, v, o, lse, ws, ws + kConstBytes, ws + windows_at, int(units.n_tiles),
            int(units.units.size() - units.n_tiles), desc->n_heads, desc->head_dim, int(desc->total_tokens),
            desc->scale, desc->causal, s};
  hipError_t e = launch_fwd(a);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "forward launch: %s", hipGetErrorString(e));
  return DCP_OK;
}

extern "C" int dcp_varlen_attn_bwd(const dcp_attn_desc* desc, const void* dout, const void* o, const float* lse,
                                   const void* q, const void* k, const void* v, void* dq, void* dk, void* dv,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if ((st = check_tensor(dout, "dout")) || (st = check_tensor(o, "o")) || (st = check_tensor(q, "q")) ||
      (st = check_tensor(k, "k")) || (st = check_tensor(v, "v")) || (st = check_tensor(dq, "dq")) ||
      (st = check_tensor(dk, "dk")) || (st = check_tensor(dv, "dv")))
    return st;
  if (!lse || reinterpret_cast<uintptr_t>(lse) % 4) return fail(DCP_ERR_INVALID, "lse is null or misaligned");
  const BwdLayout l = bwd_layout(desc);
  if (!workspace || workspace_bytes < l.total)
    return fail(DCP_ERR_WORKSPACE, "backward workspace needs %zu bytes, got %zu", l.total, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(DCP_ERR_INVALID, "workspace must be 16-byte aligned");
  if ((st = check_device())) return st;
  const UnitList units =
      build_units(desc, bwd_key_tile_rows(desc->head_dim), bwd_key_window_rows(desc->head_dim), true);
  if (units.units.empty()) return DCP_OK;
  const UnitList qunits =
      build_units(desc, bwd_query_tile_rows(desc->head_dim), bwd_query_window_rows(desc->head_dim), false);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  if ((st = upload_head({{l.units, l.windows, &units}, {l.qunits, l.qwindows, &qunits}}, workspace, s))) return st;
  BwdArgs a{dout, o, lse, q, k, v, dq, dk, dv, reinterpret_cast<float*>(ws + l.delta),
            reinterpret_cast<float*>(ws + l.lse2), ws, ws + l.units, ws + l.windows, int(units.n_tiles),
            int(units.units.size() - units.n_tiles), ws + l.qunits, ws + l.qwindows, int(qunits.n_tiles),
            int(qunits.units.size() - qunits.n_tiles),
            desc->cu_seqlens_host[desc->n_seqs], desc->n_heads, desc->head_dim, int(desc->total_tokens),
            desc->scale, desc->causal, s};
  hipError_t e = launch_bwd(a);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "backward launch: %s", hipGetErrorString(e));
  return DCP_OK;
}

extern "C" int dcp_work_list(const dcp_attn_desc* desc, int32_t pass, int32_t* units, size_t cap, size_t* n_units,
                             size_t* n_tiles, uint64_t* window_starts, size_t cap_windows, size_t* n_windows) {
  clear_error();
  int st = validate_desc(desc);
  if (st) return st;
  if (!n_units || !n_tiles || !n_windows) return fail(DCP_ERR_INVALID, "count outputs are null");
  int tile = 0, window = 0;
  const int D = desc->head_dim;
  switch (pass) {
    case 0: tile = fwd_tile_rows(D), window = fwd_window_rows(D); break;
    case 1: tile = bwd_key_tile_rows(D), window = bwd_key_window_rows(D); break;
    case 2: tile = bwd_query_tile_rows(D), window = bwd_query_window_rows(D); break;
    default: return fail(DCP_ERR_INVALID, "pass must be 0 (forward), 1 (dK/dV) or 2 (dQ)");
  }
  const UnitList l = build_units(desc, tile, window, pass == 1);
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
  int32_t cu[2] = {0, int32_t(max_len)};
  dcp_attn_desc d{1, cu, max_len, o->n_heads, o->head_dim, 1.f, o->causal};
  const size_t fw = fwd_workspace_bytes(&d);
  l.ws_bytes = std::max(fw, bwd_layout(&d).total);
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
  hipEvent_t ev[3] = {nullptr, nullptr, nullptr};
  for (auto& e : ev) {
    if (hipEventCreate(&e) != hipSuccess) {
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
    std::vector<float> tf, tb;
    for (int32_t r = 0; r < opts->warmup + opts->reps && result == DCP_OK; ++r) {
      (void)hipEventRecord(ev[0], s);
      result = dcp_varlen_attn_fwd(&d, t[0], t[1], t[2], t[3], lse, aws, l.ws_bytes, stream);
      if (result) break;
      (void)hipEventRecord(ev[1], s);
      result = dcp_varlen_attn_bwd(&d, t[4], t[3], lse, t[0], t[1], t[2], t[5], t[6], t[7], aws, l.ws_bytes, stream);
      if (result) break;
      (void)hipEventRecord(ev[2], s);
      if (hipEventSynchronize(ev[2]) != hipSuccess) {
        result = fail(DCP_ERR_HIP, "profile run failed: %s", hipGetErrorString(hipGetLastError()));
        break;
      }
      if (r >= opts->warmup) {
        float a = 0.f, b = 0.f;
        (void)hipEventElapsedTime(&a, ev[0], ev[1]);
        (void)hipEventElapsedTime(&b, ev[1], ev[2]);
        tf.push_back(a);
        tb.push_back(b);
      }
    }
    if (result) break;
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
