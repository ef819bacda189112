// Host-only driver for sanitizer runs (AddressSanitizer + UndefinedBehavior-
// Sanitizer) of libdcp's host code: the planner and schedule replay
// (dcp_plan.cpp), the work-list builder and descriptor validation
// (work_list.cpp) and the error messages (dcp_error.cpp).  No HIP: it is
// linked from those sources alone.  Reads whitespace-separated cases from
// stdin and prints one result line per case; tests/test_sanitize_host.py
// builds it with the sanitizers on and compares its output with the oracle
// and with the production library.
//
// Case formats (all integers):
//   P n_seqs lens.. n_batches has_offs [offs..] n_rows L T_C M_C
//     [seq t_f t_b m m_inp].. budget n_sp sp.. b_max n_heads hidden alpha
//     beta g_min g_max mode flags
//   S <same as P> n_devices bucket_sp iter_sync_ns
//   W n_seqs cu.. total_tokens n_heads head_dim causal scale_milli pass
//   B n_seqs cu.. total_tokens n_heads head_dim causal scale_milli
//   U n_seqs cu.. total_tokens n_heads head_dim causal scale_milli kind
//     (kind 0: per-call forward workspace, 1: per-call backward, 2: prepared batch)
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "dcp.h"
#include "work_list.h"

namespace {

bool rd(long long* x) { return std::scanf("%lld", x) == 1; }
long long need() {
  long long x = 0;
  if (!rd(&x)) {
    std::fprintf(stderr, "truncated input\n");
    std::exit(2);
  }
  return x;
}

struct PlanCase {
  std::vector<int64_t> lens;
  std::vector<int32_t> offs;
  bool has_offs = false;
  int32_t n_batches = 0;
  std::vector<dcp_cost_row> rows;
  dcp_cost_table table{};
  int64_t budget = 0;
  std::vector<int32_t> sp;
  dcp_plan_opts opts{};
};

void read_plan(PlanCase& c) {
  const long long n = need();
  for (long long i = 0; i < n; ++i) c.lens.push_back(need());
  c.n_batches = int32_t(need());
  c.has_offs = need() != 0;
  if (c.has_offs)
    for (int32_t i = 0; i <= c.n_batches; ++i) c.offs.push_back(int32_t(need()));
  const long long nr = need();
  c.table.n_layers = int32_t(need());
  c.table.T_C_ns = need();
  c.table.M_C_bytes = need();
  for (long long i = 0; i < nr; ++i) {
    dcp_cost_row r;
    r.seq_len = need();
    r.t_f_ns = need();
    r.t_b_ns = need();
    r.m_bytes = need();
    r.m_inp_bytes = need();
    c.rows.push_back(r);
  }
  c.table.rows = c.rows.data();
  c.table.n_rows = int32_t(nr);
  c.budget = need();
  const long long nsp = need();
  for (long long i = 0; i < nsp; ++i) c.sp.push_back(int32_t(need()));
  c.opts.sp_cands = c.sp.data();
  c.opts.n_sp = int32_t(nsp);
  c.opts.b_max = int32_t(need());
  c.opts.n_heads = int32_t(need());
  c.opts.hidden = need();
  c.opts.a2a_alpha_ns = need();
  c.opts.link_bytes_per_ns = need();
  c.opts.g_min = int32_t(need());
  c.opts.g_max = int32_t(need());
  c.opts.mode = int32_t(need());
  c.opts.flags = int32_t(need());
}

void run_plan() {
  PlanCase c;
  read_plan(c);
  const size_t nb = size_t(c.n_batches > 0 ? c.n_batches : 1);
  const size_t L = size_t(c.table.n_layers > 0 ? c.table.n_layers : 1);
  std::vector<int32_t> sp(nb), mb(nb), ga(nb), rl(nb);
  std::vector<uint8_t> fl(nb * L);
  std::vector<int64_t> st(nb), mem(nb);
  dcp_plan_out out{sp.data(), mb.data(), ga.data(), rl.data(), fl.data(), st.data(), mem.data(), 0, 0};
  const int s = dcp_plan(c.lens.data(), int32_t(c.lens.size()), c.has_offs ? c.offs.data() : nullptr, c.n_batches,
                         &c.table, c.budget, &c.opts, &out);
  std::printf("%d", s);
  if (s == DCP_OK) {
    for (auto* v : {&sp, &mb, &ga, &rl})
      for (size_t i = 0; i < size_t(c.n_batches); ++i) std::printf(" %d", (*v)[i]);
    for (size_t i = 0; i < size_t(c.n_batches) * size_t(c.table.n_layers); ++i) std::printf(" %d", int(fl[i]));
    for (auto* v : {&st, &mem})
      for (size_t i = 0; i < size_t(c.n_batches); ++i) std::printf(" %lld", static_cast<long long>((*v)[i]));
    std::printf(" %lld %lld", static_cast<long long>(out.idle_ns), static_cast<long long>(out.makespan_ns));
  }
  std::printf("\n");
}

void run_sim() {
  PlanCase c;
  read_plan(c);
  dcp_sim_opts so{};
  so.n_devices = int32_t(need());
  so.bucket_sp = int32_t(need());
  so.iter_sync_ns = need();
  dcp_sim_result a{}, b{};
  const int s = dcp_simulate(c.lens.data(), int32_t(c.lens.size()), c.has_offs ? c.offs.data() : nullptr,
                             c.n_batches, &c.table, c.budget, &c.opts, &so, &a, &b);
  std::printf("%d", s);
  if (s == DCP_OK)
    for (const dcp_sim_result* r : {&a, &b})
      std::printf(" %lld %lld %lld %lld %lld %d", static_cast<long long>(r->iterations),
                  static_cast<long long>(r->makespan_ns), static_cast<long long>(r->time_ns),
                  static_cast<long long>(r->busy_device_ns), static_cast<long long>(r->tokens), r->bucket_sp);
  std::printf("\n");
}

void read_desc(dcp_attn_desc& d, std::vector<int32_t>& cu) {
  const long long n = need();
  for (long long i = 0; i <= n; ++i) cu.push_back(int32_t(need()));
  d.n_seqs = int32_t(n);
  d.cu_seqlens_host = cu.data();
  d.total_tokens = need();
  d.n_heads = int32_t(need());
  d.head_dim = int32_t(need());
  d.causal = int32_t(need());
  d.scale = float(need()) / 1000.f;
}

void run_worklist() {
  dcp_attn_desc d{};
  std::vector<int32_t> cu;
  read_desc(d, cu);
  const int32_t pass = int32_t(need());
  int s = dcp::validate_desc(&d);
  std::printf("%d", s);
  if (s == DCP_OK) {
    const dcp::UnitList l = dcp::build_pass(&d, pass);
    std::printf(" %zu %zu %zu", l.units.size(), l.n_tiles, l.window_starts.size() / dcp::kWindowWords);
    for (const dcp::WorkUnit& u : l.units)
      std::printf(" %d %d %d %d %d", u.row0, u.seq0, u.seqlen, int(u.rows), int(u.head));
    for (uint64_t w : l.window_starts) std::printf(" %llu", static_cast<unsigned long long>(w));
  }
  std::printf("\n");
}

void run_batch() {
  dcp_attn_desc d{};
  std::vector<int32_t> cu;
  read_desc(d, cu);
  dcp_batch_s b;
  const int s = dcp::batch_init(&d, &b);
  std::printf("%d", s);
  if (s == DCP_OK) {
    // every part lies inside the buffer, in order, without overlap
    size_t end = dcp::kConstBytes;
    bool ok = true;
    for (int p = 0; p < 3; ++p) {
      ok = ok && b.units_at[p] >= end;
      end = b.units_at[p] + b.pass[p].units.size() * sizeof(dcp::WorkUnit);
      ok = ok && b.windows_at[p] >= end;
      end = b.windows_at[p] + b.pass[p].window_starts.size() * sizeof(uint64_t);
    }
    const size_t per_row = size_t(4) * size_t(d.n_heads) * size_t(d.total_tokens);
    ok = ok && b.lse2_at >= end && b.delta_at >= b.lse2_at + per_row && b.total >= b.delta_at + per_row;
    std::printf(" %d %zu", int(ok), b.total);
  }
  std::printf("\n");
}

// The work-list upload as the device would receive it: plan_upload's
// segments filled on the host and copied into an image of the list area
// (pre-filled with 0xAB); then every part must sit at its offset, the bytes
// between the parts of a segment must be zero and everything outside the
// segments must be untouched.
void run_upload() {
  dcp_attn_desc d{};
  std::vector<int32_t> cu;
  read_desc(d, cu);
  const int kind = int(need());
  const int s = dcp::validate_desc(&d);
  std::printf("%d", s);
  if (s != DCP_OK) {
    std::printf("\n");
    return;
  }
  dcp::UnitList l0, l1;
  dcp_batch_s b;
  std::vector<dcp::ListAt> lists;
  size_t area = 0;
  if (kind == 0) {
    const dcp::FwdLayout f = dcp::fwd_layout(&d);
    l0 = dcp::build_pass(&d, dcp::kPassFwd);
    lists = {{f.units, f.windows, &l0}};
    area = f.total;
  } else if (kind == 1) {
    const dcp::BwdLayout bl = dcp::bwd_layout(&d);
    l0 = dcp::build_pass(&d, dcp::kPassDkdv);
    l1 = dcp::build_pass(&d, dcp::kPassDq);
    lists = {{bl.units, bl.windows, &l0}, {bl.qunits, bl.qwindows, &l1}};
    area = bl.lse2;
  } else {
    if (dcp::batch_init(&d, &b) != DCP_OK) std::exit(3);
    for (int p = 0; p < 3; ++p) lists.push_back({b.units_at[p], b.windows_at[p], &b.pass[p]});
    area = b.lse2_at;
  }
  const dcp::UploadPlan u = dcp::plan_upload(lists.data(), lists.size());
  std::vector<unsigned char> buf(u.bytes), img(area, 0xAB), inside(area, 0);
  dcp::fill_segments(u, buf.data());
  size_t off = 0;
  bool ok = true;
  for (const dcp::UploadSegment& g : u.segs) {
    ok = ok && g.end <= area && g.at < g.end;
    if (!ok) break;
    std::memcpy(img.data() + g.at, buf.data() + off, g.end - g.at);
    std::memset(inside.data() + g.at, 1, g.end - g.at);
    off += g.end - g.at;
  }
  ok = ok && off == u.bytes;
  if (ok) {
    unsigned char head[dcp::kConstBytes];
    dcp::const_head(head);
    ok = std::memcmp(img.data(), head, dcp::kConstBytes) == 0;
    for (const dcp::UploadPart& p : u.parts) {
      if (p.src) ok = ok && std::memcmp(img.data() + p.at, p.src, p.bytes) == 0;
      std::memset(inside.data() + p.at, 2, p.bytes);
    }
    for (size_t i = 0; i < area && ok; ++i)
      ok = inside[i] == 2 || (inside[i] == 1 ? img[i] == 0 : img[i] == 0xAB);
  }
  size_t part_bytes = 0;
  for (const dcp::UploadPart& p : u.parts) part_bytes += p.bytes;
  std::printf(" %d %zu %zu %zu %zu\n", int(ok), u.segs.size(), u.bytes, part_bytes, area);
}

}  // namespace

int main() {
  char op[4];
  while (std::scanf("%3s", op) == 1) {
    switch (op[0]) {
      case 'P': run_plan(); break;
      case 'S': run_sim(); break;
      case 'W': run_worklist(); break;
      case 'B': run_batch(); break;
      case 'U': run_upload(); break;
      default: std::fprintf(stderr, "unknown case %s\n", op); return 2;
    }
  }
  return 0;
}
