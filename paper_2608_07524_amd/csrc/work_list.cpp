// Host-side work lists of the attention kernels (see work_list.h).
#include "work_list.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>

#include "dcp_internal.h"

namespace dcp {

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

UnitList build_pass(const dcp_attn_desc* d, int32_t pass) {
  const int D = d->head_dim;
  switch (pass) {
    case kPassFwd: return build_units(d, fwd_tile_rows(D), fwd_window_rows(D), false);
    case kPassDkdv: return build_units(d, bwd_key_tile_rows(D), bwd_key_window_rows(D), true);
    default: return build_units(d, bwd_query_tile_rows(D), bwd_query_window_rows(D), false);
  }
}

void const_head(unsigned char (&head)[kConstBytes]) {
  std::memset(head, 0, sizeof head);
  const uint16_t one = 0x3F80;  // bf16 1.0
  std::memcpy(head + kConstOnes * 2, &one, sizeof one);
  const float inf = std::numeric_limits<float>::infinity();
  std::memcpy(head + kConstInf * 2, &inf, sizeof inf);
}

FwdLayout fwd_layout(const dcp_attn_desc* d) {
  const int t = fwd_tile_rows(d->head_dim);
  FwdLayout l;
  l.units = kConstBytes;
  l.windows = l.units + list_bytes(d, t);
  l.total = l.windows + window_bytes(d, t);
  return l;
}

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

UploadPlan plan_upload(const ListAt* lists, size_t n_lists) {
  UploadPlan u;
  u.parts.reserve(1 + 2 * n_lists);
  u.parts.push_back({0, kConstBytes, nullptr});
  for (size_t i = 0; i < n_lists; ++i) {
    const UnitList& x = *lists[i].list;
    if (!x.units.empty()) u.parts.push_back({lists[i].units_at, x.units.size() * sizeof(WorkUnit), x.units.data()});
    if (!x.window_starts.empty())
      u.parts.push_back({lists[i].windows_at, x.window_starts.size() * sizeof(uint64_t), x.window_starts.data()});
  }
  std::sort(u.parts.begin(), u.parts.end(), [](const UploadPart& p, const UploadPart& q) { return p.at < q.at; });
  for (const UploadPart& p : u.parts) {  // the parts do not overlap
    if (!u.segs.empty() && p.at - u.segs.back().end <= kMergeGap)
      u.segs.back().end = p.at + p.bytes;
    else
      u.segs.push_back({p.at, p.at + p.bytes});
  }
  for (const UploadSegment& g : u.segs) u.bytes += g.end - g.at;
  return u;
}

void fill_segments(const UploadPlan& u, unsigned char* buf) {
  size_t off = 0;  // host offset of the current segment
  size_t k = 0;    // next part
  for (const UploadSegment& g : u.segs) {
    size_t at = g.at;
    for (; k < u.parts.size() && u.parts[k].at < g.end; ++k) {
      const UploadPart& p = u.parts[k];
      unsigned char* out = buf + off + (p.at - g.at);
      std::memset(buf + off + (at - g.at), 0, p.at - at);
      if (p.src)
        std::memcpy(out, p.src, p.bytes);
      else
        const_head(*reinterpret_cast<unsigned char(*)[kConstBytes]>(out));
      at = p.at + p.bytes;
    }
    off += g.end - g.at;
  }
}

int batch_init(const dcp_attn_desc* desc, dcp_batch_s* b) {
  int st = validate_desc(desc);
  if (st) return st;
  b->desc = *desc;
  b->cu.assign(desc->cu_seqlens_host, desc->cu_seqlens_host + desc->n_seqs + 1);
  b->desc.cu_seqlens_host = b->cu.data();
  size_t off = kConstBytes;
  for (int32_t p = 0; p < 3; ++p) {
    b->pass[p] = build_pass(&b->desc, p);
    b->units_at[p] = off;
    off += align_up(std::max<size_t>(1, b->pass[p].units.size()) * sizeof(WorkUnit));
    b->windows_at[p] = off;
    off += align_up(std::max<size_t>(1, b->pass[p].window_starts.size()) * sizeof(uint64_t));
  }
  const size_t per_row = align_up(size_t(4) * size_t(desc->n_heads) * size_t(desc->total_tokens));
  b->lse2_at = off;
  b->delta_at = off + per_row;
  b->total = off + 2 * per_row;
  b->uploaded = nullptr;
  b->device = -1;
  return DCP_OK;
}

}  // namespace dcp
