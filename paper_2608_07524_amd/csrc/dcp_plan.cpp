// Host-side DCP planner: DCP-intra (Sec. 3.4, Eqs. (4)-(6), Algorithm 1),
// DCP-inter (Sec. 3.3, Eq. (3)) and the accumulation bounds of Appendix C.
//
// Pure integer arithmetic (int64 values, __int128 for exact products and
// comparisons), no device code, reentrant.  Every intermediate quantity is
// checked to fit int64; an overflow is reported as DCP_ERR_INVALID.
//
// Model (per layer, one GPU, micro-batch 1, from the cost table):
//   per batch i: t_f1, t_b1, m1, m_inp1 = sums over its sequences of the row
//   with the smallest tabulated length >= the sequence length (grouping by
//   similar size, Sec. 3.1), S_i = its token count.
//   candidate (p, b): comm c = 0 for p = 1, else 4*(alpha + ceil(2*b*S_i*h /
//   (p^2*beta))) -- four Ulysses all-to-alls per layer each way, each link of
//   a fully connected node carrying 1/p^2 of the activations;
//   t_f = ceil(b*t_f1/p) + c, t_b = ceil(b*t_b1/p) + c,
//   m = ceil(b*m1/p), m_inp = ceil(b*m_inp1/p), base = L*m_inp + M_C.
//   Eq. (6): memory with r recomputed layers = (L-r)*m + base; the smallest
//   r that fits is r = L - min(L, floor((M - base)/m)) (r = 0 when m = 0).
//   Eqs. (4)-(5): T = L*(t_f + t_b) + r*t_f + T_C.
//   Selection: maximal Eq. (1) throughput b*S_i/(p*T) (S_i is common to a
//   batch's candidates), ties to smaller p then smaller b.  DCP-inter fixes
//   r = L (full recomputation) and needs base <= M.
//   Accumulation (Eq. (3)): minimise sum_i (C - g_i*T_i) with C = max_i
//   g_i*T_i <= G_max*max_i T_i.  For a fixed C the minimiser is g_i =
//   floor(C/T_i), and C is a multiple of some T_j, so all such multiples are
//   scanned; ties go to the smallest C.  Then, if max_i g_i < G_min, every
//   g_i is multiplied by ceil(G_min / max_i g_i).
#include <algorithm>
#include <cstring>
#include <vector>

#include "dcp_internal.h"

namespace {

using i128 = __int128;
constexpr int64_t kI64Max = INT64_MAX;
constexpr int64_t kMaxAccumCandidates = int64_t(1) << 22;

struct Overflow {};

inline int64_t chk(i128 x) {
  if (x > i128(kI64Max) || x < -i128(kI64Max) - 1) throw Overflow{};
  return int64_t(x);
}
inline int64_t ceil_div(int64_t a, int64_t b) { return a / b + ((a % b) != 0); }

struct Unit {
  int64_t tokens = 0, t_f = 0, t_b = 0, m = 0, m_inp = 0;
};

struct Choice {
  int32_t p = 0, b = 0, r = 0;
  int64_t T = 0, mem = 0;
};

const int32_t kDefaultSp[4] = {1, 2, 4, 8};

}  // namespace

extern "C" void dcp_plan_opts_default(dcp_plan_opts* o) {
  if (!o) return;
  o->sp_cands = kDefaultSp;
  o->n_sp = 4;
  o->b_max = 64;
  o->n_heads = 16;
  o->hidden = 1152;
  o->a2a_alpha_ns = 10000;
  o->link_bytes_per_ns = 153;
  o->g_min = 1;
  o->g_max = 4;
  o->mode = DCP_PLAN_INTRA;
  o->flags = 0;
}

namespace {

int validate(const int64_t* seq_lens, int32_t n_seqs, const int32_t* offs, int32_t n_batches,
             const dcp_cost_table* t, int64_t budget, const dcp_plan_opts& o) {
  using dcp::fail;
  if (n_batches < 1 || n_seqs < 1) return fail(DCP_ERR_INVALID, "need at least one batch and one sequence");
  if (!seq_lens) return fail(DCP_ERR_INVALID, "seq_lens is null");
  if (!offs) {
    if (n_batches != n_seqs) return fail(DCP_ERR_INVALID, "without batch offsets every sequence is its own batch");
  } else {
    if (offs[0] != 0 || offs[n_batches] != n_seqs)
      return fail(DCP_ERR_INVALID, "batch offsets must run from 0 to the sequence count");
    for (int32_t i = 0; i < n_batches; ++i)
      if (offs[i + 1] <= offs[i]) return fail(DCP_ERR_INVALID, "every batch needs at least one sequence");
  }
  for (int32_t i = 0; i < n_seqs; ++i)
    if (seq_lens[i] < 1) return fail(DCP_ERR_INVALID, "sequence lengths must be positive (index %d)", i);
  if (budget < 0) return fail(DCP_ERR_INVALID, "memory budget must be non-negative");
  if (o.n_sp < 1 || !o.sp_cands) return fail(DCP_ERR_INVALID, "need at least one sequence-parallel size");
  for (int32_t i = 0; i < o.n_sp; ++i)
    if (o.sp_cands[i] <= (i ? o.sp_cands[i - 1] : 0))
      return fail(DCP_ERR_INVALID, "sequence-parallel sizes must be positive and strictly increasing");
  if (o.b_max < 1 || o.n_heads < 1 || o.hidden < 0 || o.a2a_alpha_ns < 0 || o.link_bytes_per_ns < 1 ||
      o.g_min < 1 || o.g_max < 1 || (o.mode != DCP_PLAN_INTER && o.mode != DCP_PLAN_INTRA) ||
      (o.flags & ~(DCP_PLAN_FLAG_MIN_TIME | DCP_PLAN_FLAG_NO_HEAD_FILTER)) != 0)
    return fail(DCP_ERR_INVALID, "bad planner options");
  if (!t || t->n_rows < 1 || !t->rows || t->n_layers < 1 || t->T_C_ns < 0 || t->M_C_bytes < 0)
    return fail(DCP_ERR_TABLE, "cost table needs rows, at least one layer and non-negative constants");
  for (int32_t i = 0; i < t->n_rows; ++i) {
    const dcp_cost_row& r = t->rows[i];
    if (r.seq_len <= (i ? t->rows[i - 1].seq_len : 0))
      return fail(DCP_ERR_TABLE, "cost table lengths must be positive and strictly increasing (row %d)", i);
    if (r.t_f_ns < 0 || r.t_b_ns < 0 || r.m_bytes < 0 || r.m_inp_bytes < 0)
      return fail(DCP_ERR_TABLE, "cost table entries must be non-negative (row %d)", i);
  }
  return DCP_OK;
}

// Binary search for the first row with seq_len >= s.
const dcp_cost_row* row_for(const dcp_cost_table* t, int64_t s) {
  const dcp_cost_row* lo = t->rows;
  const dcp_cost_row* hi = t->rows + t->n_rows;
  const dcp_cost_row* it =
      std::lower_bound(lo, hi, s, [](const dcp_cost_row& r, int64_t v) { return r.seq_len < v; });
  return it == hi ? nullptr : it;
}

// Per-layer costs of b copies of a batch on p devices: the Ulysses
// all-to-all term c, then t_f, t_b, m, m_inp and base = L*m_inp + M_C
// (Eq. (6) with every layer recomputed).
struct LayerCost {
  int64_t t_f, t_b, m, m_inp, base;
};
LayerCost layer_cost(const Unit& u, const dcp_cost_table* t, const dcp_plan_opts& o, int64_t p, int64_t b) {
  const int64_t L = t->n_layers;
  int64_t c = 0;
  if (p != 1) {
    int64_t vol = chk(i128(chk(i128(chk(i128(b) * u.tokens)) * o.hidden)) * 2);
    int64_t per_link = chk(i128(chk(i128(p) * p)) * o.link_bytes_per_ns);
    c = chk(i128(4) * chk(i128(o.a2a_alpha_ns) + ceil_div(vol, per_link)));
  }
  LayerCost k;
  k.t_f = chk(i128(ceil_div(chk(i128(b) * u.t_f), p)) + c);
  k.t_b = chk(i128(ceil_div(chk(i128(b) * u.t_b), p)) + c);
  k.m = ceil_div(chk(i128(b) * u.m), p);
  k.m_inp = ceil_div(chk(i128(b) * u.m_inp), p);
  k.base = chk(i128(chk(i128(L) * k.m_inp)) + t->M_C_bytes);
  return k;
}

// Eqs. (4)-(5): T = L*(t_f + t_b) + r*t_f + T_C.
int64_t step_time(const LayerCost& k, int64_t r, const dcp_cost_table* t) {
  const int64_t L = t->n_layers;
  return chk(i128(chk(i128(chk(i128(L) * chk(i128(k.t_f) + k.t_b))) + chk(i128(r) * k.t_f))) + t->T_C_ns);
}

// Returns DCP_OK and fills `best`, or an error status.
int choose(const Unit& u, const dcp_cost_table* t, int64_t budget, const dcp_plan_opts& o, int32_t batch,
           Choice* best_out) {
  const int64_t L = t->n_layers;
  bool have = false;
  Choice best;
  for (int32_t pi = 0; pi < o.n_sp; ++pi) {
    const int64_t p = o.sp_cands[pi];
    if (!(o.flags & DCP_PLAN_FLAG_NO_HEAD_FILTER) && (o.n_heads % p) != 0) continue;
    for (int64_t b = 1; b <= o.b_max; ++b) {
      const LayerCost k = layer_cost(u, t, o, p, b);
      const int64_t m = k.m, base = k.base;
      if (base > budget) continue;
      int64_t r;
      if (o.mode == DCP_PLAN_INTER) {
        r = L;
      } else {
        const int64_t kept = (m == 0) ? L : std::min<int64_t>(L, (budget - base) / m);
        r = L - kept;
      }
      const int64_t T = step_time(k, r, t);
      bool better;
      if (!have) {
        better = true;
      } else if (o.flags & DCP_PLAN_FLAG_MIN_TIME) {
        better = T < best.T;
      } else {
        // b/(p*T) > best.b/(best.p*best.T)
        better = i128(b) * best.p * best.T > i128(best.b) * p * T;
      }
      if (better) {
        have = true;
        best.p = int32_t(p);
        best.b = int32_t(b);
        best.r = int32_t(r);
        best.T = T;
        best.mem = int64_t(i128(L - r) * m + base);  // <= budget by construction
      }
    }
  }
  if (!have) return dcp::fail(DCP_ERR_INFEASIBLE, "no feasible configuration for batch %d", batch);
  *best_out = best;
  return DCP_OK;
}

// Per-batch sums of the table rows of its sequences (each sequence takes the
// row with the smallest length >= its own).
int batch_units(const int64_t* seq_lens, const int32_t* batch_offsets, int32_t n_batches, const dcp_cost_table* table,
                std::vector<Unit>* out) {
  std::vector<Unit>& units = *out;
  units.assign(static_cast<size_t>(n_batches), Unit{});
  for (int32_t i = 0; i < n_batches; ++i) {
    const int32_t lo = batch_offsets ? batch_offsets[i] : i;
    const int32_t hi = batch_offsets ? batch_offsets[i + 1] : i + 1;
    Unit& u = units[size_t(i)];
    for (int32_t s = lo; s < hi; ++s) {
      const dcp_cost_row* r = row_for(table, seq_lens[s]);
      if (!r)
        return dcp::fail(DCP_ERR_TABLE, "sequence length %lld exceeds the cost table",
                         static_cast<long long>(seq_lens[s]));
      u.tokens = chk(i128(u.tokens) + seq_lens[s]);
      u.t_f = chk(i128(u.t_f) + r->t_f_ns);
      u.t_b = chk(i128(u.t_b) + r->t_b_ns);
      u.m = chk(i128(u.m) + r->m_bytes);
      u.m_inp = chk(i128(u.m_inp) + r->m_inp_bytes);
    }
  }
  return DCP_OK;
}

int accumulate(const std::vector<int64_t>& T, int32_t g_min, int32_t g_max, std::vector<int64_t>* g_out,
               int64_t* idle_out, int64_t* span_out) {
  const int64_t tmax = *std::max_element(T.begin(), T.end());
  const int64_t bound = chk(i128(g_max) * tmax);
  i128 count = 0;
  for (int64_t t : T) count += bound / t - ceil_div(tmax, t) + 1;
  if (count > kMaxAccumCandidates) return dcp::fail(DCP_ERR_INVALID, "accumulation search too large");
  std::vector<int64_t> cands;
  cands.reserve(size_t(count));
  for (int64_t t : T)
    for (int64_t k = ceil_div(tmax, t); k <= bound / t; ++k) cands.push_back(k * t);
  std::sort(cands.begin(), cands.end());
  cands.erase(std::unique(cands.begin(), cands.end()), cands.end());
  i128 best_idle = -1;
  int64_t best_c = 0;
  for (int64_t C : cands) {
    i128 idle = 0;
    for (int64_t t : T) idle += C % t;
    if (best_idle < 0 || idle < best_idle) {
      best_idle = idle;
      best_c = C;
    }
  }
  std::vector<int64_t>& g = *g_out;
  g.resize(T.size());
  int64_t gmax = 0;
  for (size_t i = 0; i < T.size(); ++i) {
    g[i] = best_c / T[i];
    gmax = std::max(gmax, g[i]);
  }
  if (gmax < g_min) {
    const int64_t f = ceil_div(g_min, gmax);
    for (auto& x : g) x *= f;
  }
  int64_t span = 0;
  for (size_t i = 0; i < T.size(); ++i) span = std::max(span, chk(i128(g[i]) * T[i]));
  i128 idle = 0;
  for (size_t i = 0; i < T.size(); ++i) idle += i128(span) - i128(g[i]) * T[i];
  *idle_out = chk(idle);
  *span_out = span;
  return DCP_OK;
}

}  // namespace

extern "C" int dcp_plan(const int64_t* seq_lens, int32_t n_seqs, const int32_t* batch_offsets, int32_t n_batches,
                        const dcp_cost_table* table, int64_t hbm_budget_bytes, const dcp_plan_opts* opts_in,
                        dcp_plan_out* out) {
  dcp::clear_error();
  try {
    dcp_plan_opts o;
    if (opts_in) {
      o = *opts_in;
    } else {
      dcp_plan_opts_default(&o);
    }
    if (!out || !out->sp_size || !out->micro_batch || !out->grad_accum || !out->recompute_layers ||
        !out->recompute_flags)
      return dcp::fail(DCP_ERR_INVALID, "plan output arrays must not be null");
    int st = validate(seq_lens, n_seqs, batch_offsets, n_batches, table, hbm_budget_bytes, o);
    if (st != DCP_OK) return st;

    std::vector<Unit> units;
    st = batch_units(seq_lens, batch_offsets, n_batches, table, &units);
    if (st != DCP_OK) return st;
    std::vector<Choice> ch(static_cast<size_t>(n_batches));
    std::vector<int64_t> T(static_cast<size_t>(n_batches));
    for (int32_t i = 0; i < n_batches; ++i) {
      st = choose(units[size_t(i)], table, hbm_budget_bytes, o, i, &ch[size_t(i)]);
      if (st != DCP_OK) return st;
      T[size_t(i)] = ch[size_t(i)].T;
    }
    if (*std::min_element(T.begin(), T.end()) == 0)
      return dcp::fail(DCP_ERR_TABLE, "a batch has zero step time; the cost table is empty of cost");
    std::vector<int64_t> g;
    int64_t idle = 0, span = 0;
    st = accumulate(T, o.g_min, o.g_max, &g, &idle, &span);
    if (st != DCP_OK) return st;
    for (const auto& x : g)
      if (x > INT32_MAX) return dcp::fail(DCP_ERR_INVALID, "accumulation steps exceed int32");

    const int32_t L = table->n_layers;
    for (int32_t i = 0; i < n_batches; ++i) {
      const Choice& c = ch[size_t(i)];
      out->sp_size[i] = c.p;
      out->micro_batch[i] = c.b;
      out->grad_accum[i] = int32_t(g[size_t(i)]);
      out->recompute_layers[i] = c.r;
      for (int32_t l = 0; l < L; ++l) out->recompute_flags[size_t(i) * size_t(L) + size_t(l)] = l < c.r ? 1 : 0;
      if (out->step_time_ns) out->step_time_ns[i] = c.T;
      if (out->mem_bytes) out->mem_bytes[i] = c.mem;
    }
    out->idle_ns = idle;
    out->makespan_ns = span;
    return DCP_OK;
  } catch (const Overflow&) {
    return dcp::fail(DCP_ERR_INVALID, "int64 overflow in planner arithmetic");
  } catch (...) {
    return dcp::fail(DCP_ERR_INVALID, "planner failed (out of host memory)");
  }
}

// ---------------------------------------------------------------------------
// Schedule replay: DCP against bucket parallelism over a stream of batches
// on W devices (the comparison of Sec. 4.2: throughput, Eq. (1), and the
// imbalance ratio, the share of device time spent waiting).
//
// DCP: every batch takes the planner's (p_i, b_i, r_i, T_i); batches join
// the current iteration in stream order while they fit the devices left
// (Eq. (1)'s sum_i p_i <= W): of the first kSimWindow batches not yet
// placed, each that fits joins the iteration and each that does not waits
// for a later one, keeping its place in the stream (devices still left over
// wait out the iteration); the iteration's
// accumulation steps g_i follow Eq. (3) with the bounds of Appendix C.
// Bucket parallelism (Sec. 4.1 baseline, Sec. 2.4): one fixed p for every
// batch, floor(W/p) batches per iteration in stream order, no accumulation,
// full recomputation, and a static batch size per batch -- the largest b
// whose step time does not exceed that of the slowest batch of the stream at
// b = 1 (long batches stay at 1, short ones grow), within memory.
// Per iteration: makespan = max_i g_i*T_i, busy device time sum_i
// p_i*g_i*T_i, tokens sum_i g_i*b_i*S_i, time = makespan + sync.

namespace {

// batches an iteration looks at when filling its devices
constexpr int64_t kSimWindow = 64;

int sim_dcp(const std::vector<Unit>& units, const dcp_cost_table* t, int64_t budget, const dcp_plan_opts& o,
            int64_t W, int64_t sync, dcp_sim_result* res) {
  const size_t n = units.size();
  std::vector<Choice> ch(n);
  for (size_t i = 0; i < n; ++i) {
    int st = choose(units[i], t, budget, o, int32_t(i), &ch[i]);
    if (st != DCP_OK) return st;
    if (ch[i].p > W) return dcp::fail(DCP_ERR_INVALID, "batch %zu needs %d devices, more than W", i, ch[i].p);
    if (ch[i].T == 0) return dcp::fail(DCP_ERR_TABLE, "a batch has zero step time; the cost table is empty of cost");
  }
  *res = dcp_sim_result{};
  // batches not yet placed, in stream order
  std::vector<size_t> pending(n), rest;
  for (size_t i = 0; i < n; ++i) pending[i] = i;
  std::vector<size_t> members;
  while (!pending.empty()) {
    members.clear();
    rest.clear();
    int64_t used = 0;
    for (size_t x = 0; x < pending.size(); ++x) {
      const size_t k = pending[x];
      if (x < size_t(kSimWindow) && used + ch[k].p <= W) {
        members.push_back(k);
        used += ch[k].p;
      } else {
        rest.push_back(k);
      }
    }
    pending.swap(rest);
    std::vector<int64_t> T(members.size()), g;
    for (size_t m = 0; m < members.size(); ++m) T[m] = ch[members[m]].T;
    int64_t idle = 0, span = 0;
    int st = accumulate(T, o.g_min, o.g_max, &g, &idle, &span);
    if (st != DCP_OK) return st;
    i128 busy = 0, tokens = 0;
    for (size_t m = 0; m < members.size(); ++m) {
      const size_t k = members[m];
      busy += i128(ch[k].p) * g[m] * ch[k].T;
      tokens += i128(g[m]) * ch[k].b * units[k].tokens;
    }
    res->iterations += 1;
    res->makespan_ns = chk(i128(res->makespan_ns) + span);
    res->time_ns = chk(i128(res->time_ns) + span + sync);
    res->busy_device_ns = chk(i128(res->busy_device_ns) + busy);
    res->tokens = chk(i128(res->tokens) + tokens);
  }
  return DCP_OK;
}

int sim_bucket(const std::vector<Unit>& units, const dcp_cost_table* t, int64_t budget, const dcp_plan_opts& o,
               int64_t W, int64_t sync, int32_t p_req, dcp_sim_result* res) {
  const int64_t L = t->n_layers;
  const size_t n = units.size();
  auto fits_at_one = [&](int64_t p) {
    for (const Unit& u : units)
      if (layer_cost(u, t, o, p, 1).base > budget) return false;
    return true;
  };
  int64_t p = p_req;
  if (p == 0) {
    for (int32_t pi = 0; pi < o.n_sp && p == 0; ++pi) {
      const int64_t c = o.sp_cands[pi];
      if (c > W) break;
      if (!(o.flags & DCP_PLAN_FLAG_NO_HEAD_FILTER) && (o.n_heads % c) != 0) continue;
      if (fits_at_one(c)) p = c;
    }
    if (p == 0) return dcp::fail(DCP_ERR_INFEASIBLE, "no sequence-parallel size fits every batch at micro-batch 1");
  } else {
    if (p > W) return dcp::fail(DCP_ERR_INVALID, "bucket sequence-parallel size exceeds W");
    if (!fits_at_one(p)) return dcp::fail(DCP_ERR_INFEASIBLE, "a batch does not fit at the bucket sequence-parallel size");
  }
  int64_t target = 0;
  for (const Unit& u : units) target = std::max(target, step_time(layer_cost(u, t, o, p, 1), L, t));
  if (target == 0) return dcp::fail(DCP_ERR_TABLE, "a batch has zero step time; the cost table is empty of cost");
  std::vector<int64_t> b(n), T(n);
  for (size_t i = 0; i < n; ++i) {
    b[i] = 1;
    T[i] = step_time(layer_cost(units[i], t, o, p, 1), L, t);
    for (int64_t bb = 2; bb <= o.b_max; ++bb) {
      const LayerCost k = layer_cost(units[i], t, o, p, bb);
      const int64_t Tb = step_time(k, L, t);
      if (k.base > budget || Tb > target) break;  // both grow with b
      b[i] = bb;
      T[i] = Tb;
    }
  }
  *res = dcp_sim_result{};
  res->bucket_sp = int32_t(p);
  const size_t per = size_t(W / p);
  for (size_t i = 0; i < n; i += per) {
    const size_t j = std::min(n, i + per);
    int64_t span = 0;
    i128 busy = 0, tokens = 0;
    for (size_t k = i; k < j; ++k) {
      span = std::max(span, T[k]);
      busy += i128(p) * T[k];
      tokens += i128(b[k]) * units[k].tokens;
    }
    res->iterations += 1;
    res->makespan_ns = chk(i128(res->makespan_ns) + span);
    res->time_ns = chk(i128(res->time_ns) + span + sync);
    res->busy_device_ns = chk(i128(res->busy_device_ns) + busy);
    res->tokens = chk(i128(res->tokens) + tokens);
  }
  return DCP_OK;
}

}  // namespace

extern "C" int dcp_simulate(const int64_t* seq_lens, int32_t n_seqs, const int32_t* batch_offsets, int32_t n_batches,
                            const dcp_cost_table* table, int64_t hbm_budget_bytes, const dcp_plan_opts* opts_in,
                            const dcp_sim_opts* sim, dcp_sim_result* dcp_out, dcp_sim_result* bucket_out) {
  dcp::clear_error();
  try {
    dcp_plan_opts o;
    if (opts_in) {
      o = *opts_in;
    } else {
      dcp_plan_opts_default(&o);
    }
    if (!sim || !dcp_out || !bucket_out) return dcp::fail(DCP_ERR_INVALID, "simulation options and results must not be null");
    if (sim->n_devices < 1 || sim->bucket_sp < 0 || sim->iter_sync_ns < 0)
      return dcp::fail(DCP_ERR_INVALID, "need n_devices >= 1, bucket_sp >= 0 and iter_sync_ns >= 0");
    int st = validate(seq_lens, n_seqs, batch_offsets, n_batches, table, hbm_budget_bytes, o);
    if (st != DCP_OK) return st;
    std::vector<Unit> units;
    st = batch_units(seq_lens, batch_offsets, n_batches, table, &units);
    if (st != DCP_OK) return st;
    dcp_sim_result a{}, b{};
    st = sim_dcp(units, table, hbm_budget_bytes, o, sim->n_devices, sim->iter_sync_ns, &a);
    if (st != DCP_OK) return st;
    st = sim_bucket(units, table, hbm_budget_bytes, o, sim->n_devices, sim->iter_sync_ns, sim->bucket_sp, &b);
    if (st != DCP_OK) return st;
    *dcp_out = a;
    *bucket_out = b;
    return DCP_OK;
  } catch (const Overflow&) {
    return dcp::fail(DCP_ERR_INVALID, "int64 overflow in simulation arithmetic");
  } catch (...) {
    return dcp::fail(DCP_ERR_INVALID, "simulation failed (out of host memory)");
  }
}
