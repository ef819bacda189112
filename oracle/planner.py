"""Integer oracle for the DCP planner (DCP-intra, DCP-inter and the
gradient-accumulation search), plus exhaustive brute-force searches.

TEST INFRASTRUCTURE ONLY. This module is imported by ``tests/`` (and may be
used by ``bench.py``'s CPU baseline); the product planner is an independent
C++ implementation behind the C ABI and shares no code with this file.

Every quantity is a Python int (nanoseconds, bytes).  Comparisons of
throughputs use exact cross-multiplication, so the result is a pure function
of the integer inputs and can be compared bit for bit.  Every intermediate
result is checked to fit a signed 64-bit integer, mirroring the product's
overflow rule.

Sources in the paper and the readings taken where it is silent or garbled
-------------------------------------------------------------------------
* Problem statement (Sec. 3.2): n batches d_i of sequence length s_i per
  iteration; choose batch size b_i, sequence-parallel size p_i (and, Sec.
  3.3/3.4, accumulation steps g_i and recomputed layers r_i) per batch.
  Eq. (1) maximises per-GPU throughput b_i*s_i / (p_i*T(d_i)); Eq. (2)/(3)
  minimise idle time against the slowest batch.
* Time and memory model (Sec. 3.4, Eqs. (4)-(6)):
      T = T_f + T_b + T_f' + T_C,   T_f' = r * t_f
      M = (L - r) * m + L * m_inp + M_C
  with per-layer forward time t_f, backward time t_b, stashed activations m
  and layer input m_inp.  T_f = L*t_f and T_b = L*t_b.
* Dual-layer profile (Sec. 3.5): one measured layer gives t_f, t_b, m; the
  model-wide estimate with full recomputation is L*(2 t_f + t_b) + T_C and
  the memory is Eq. (6) at r = L.
* Algorithm 1 (DCP-intra): for every profiled (b, p) find the smallest r
  that fits the memory capacity M, compute the time, and keep the best.
  Reading: the printed loop counts the layers that are *not* recomputed and
  compares raw times; here r is the number of recomputed layers (as in
  Eq. (5)), infeasible (b, p) are skipped, and candidates are compared by
  Eq. (1) throughput as the text of Sec. 3.4 says (the literal raw-time
  objective is available with ``FLAG_MIN_TIME``).  Ties go to the smaller p,
  then the smaller b.
* DCP-inter (Sec. 3.3): the best (b, p) per length from the profile with
  full recomputation (r = L), then accumulation steps g_i minimising
  Eq. (3), sum_i (max_j g_j T_j - g_i T_i); all combinations are searched.
  Appendix C bounds the search: the iteration may last at most G_max times
  the slowest batch, and if every g_i is below G_min all are scaled up by
  ceil(G_min / max_i g_i).  Ties go to the shortest iteration.
* Grouping (Sec. 3.1, sequences are grouped into groups of similar size and
  each group is profiled): each sequence takes the profile row with the
  smallest tabulated length >= its own; a pack of several sequences sums
  their rows.
* Candidate costs: the table holds one-GPU (b = 1, p = 1) rows.  Ulysses
  splits heads for attention and tokens elsewhere (Sec. 6.1), so times and
  memory scale as ceil(b*x/p); for p > 1 each layer adds four all-to-alls
  in forward and four in backward, each alpha + ceil(b*S*hidden*2 /
  (p^2*beta)) ns for a pack of S tokens (per-link bound on a fully connected
  node).  Only sizes p dividing the head count are used (after the all-to-all
  each device holds H/p heads) unless ``FLAG_NO_HEAD_FILTER`` is set.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from itertools import product
from typing import List, Optional, Sequence

INT64_MAX = (1 << 63) - 1

OK = 0
ERR_INVALID = -1
ERR_UNSUPPORTED = -2
ERR_HIP = -3
ERR_WORKSPACE = -4
ERR_INFEASIBLE = -5
ERR_TABLE = -6

FLAG_MIN_TIME = 1
FLAG_NO_HEAD_FILTER = 2
_KNOWN_FLAGS = FLAG_MIN_TIME | FLAG_NO_HEAD_FILTER

MODE_INTER = 0
MODE_INTRA = 1

# Upper bound on the number of iteration-length candidates the accumulation
# search may visit.
MAX_ACCUM_CANDIDATES = 1 << 22


class PlanError(Exception):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


@dataclass(frozen=True)
class CostRow:
    seq_len: int
    t_f_ns: int
    t_b_ns: int
    m_bytes: int
    m_inp_bytes: int


@dataclass(frozen=True)
class CostTable:
    rows: Sequence[CostRow]
    n_layers: int
    T_C_ns: int
    M_C_bytes: int


@dataclass(frozen=True)
class PlanOpts:
    sp_cands: Sequence[int] = (1, 2, 4, 8)
    b_max: int = 64
    n_heads: int = 16
    hidden: int = 1152
    a2a_alpha_ns: int = 10_000
    link_bytes_per_ns: int = 153
    g_min: int = 1
    g_max: int = 4
    mode: int = MODE_INTRA
    flags: int = 0


@dataclass
class Plan:
    sp_size: List[int] = field(default_factory=list)
    micro_batch: List[int] = field(default_factory=list)
    grad_accum: List[int] = field(default_factory=list)
    recompute_layers: List[int] = field(default_factory=list)
    recompute_flags: List[int] = field(default_factory=list)
    step_time_ns: List[int] = field(default_factory=list)
    mem_bytes: List[int] = field(default_factory=list)
    idle_ns: int = 0
    makespan_ns: int = 0


def _fit(x: int) -> int:
    if x > INT64_MAX or x < -INT64_MAX - 1:
        raise PlanError(ERR_INVALID, "int64 overflow in planner arithmetic")
    return x


def _ceil_div(a: int, b: int) -> int:
    return -((-a) // b)


# --------------------------------------------------------------------------
# validation (shared order of checks with the product, so error codes agree)
# --------------------------------------------------------------------------

def _validate(seq_lens, batch_offsets, n_batches, table, budget, opts):
    if n_batches < 1 or len(seq_lens) < 1:
        raise PlanError(ERR_INVALID, "need at least one batch and one sequence")
    if batch_offsets is None:
        if n_batches != len(seq_lens):
            raise PlanError(ERR_INVALID, "without batch offsets every sequence is its own batch")
    else:
        if len(batch_offsets) != n_batches + 1 or batch_offsets[0] != 0 or batch_offsets[-1] != len(seq_lens):
            raise PlanError(ERR_INVALID, "batch offsets must run from 0 to the sequence count")
        for i in range(n_batches):
            if batch_offsets[i + 1] <= batch_offsets[i]:
                raise PlanError(ERR_INVALID, "every batch needs at least one sequence")
    for s in seq_lens:
        if s < 1:
            raise PlanError(ERR_INVALID, "sequence lengths must be positive")
    if budget < 0:
        raise PlanError(ERR_INVALID, "memory budget must be non-negative")
    o = opts
    if len(o.sp_cands) < 1:
        raise PlanError(ERR_INVALID, "need at least one sequence-parallel size")
    prev = 0
    for p in o.sp_cands:
        if p <= prev:
            raise PlanError(ERR_INVALID, "sequence-parallel sizes must be positive and strictly increasing")
        prev = p
    if (o.b_max < 1 or o.n_heads < 1 or o.hidden < 0 or o.a2a_alpha_ns < 0 or o.link_bytes_per_ns < 1
            or o.g_min < 1 or o.g_max < 1 or o.mode not in (MODE_INTER, MODE_INTRA)
            or (o.flags & ~_KNOWN_FLAGS) != 0):
        raise PlanError(ERR_INVALID, "bad planner options")
    if len(table.rows) < 1 or table.n_layers < 1 or table.T_C_ns < 0 or table.M_C_bytes < 0:
        raise PlanError(ERR_TABLE, "cost table needs rows, at least one layer and non-negative constants")
    prev = 0
    for r in table.rows:
        if r.seq_len <= prev:
            raise PlanError(ERR_TABLE, "cost table lengths must be positive and strictly increasing")
        if r.t_f_ns < 0 or r.t_b_ns < 0 or r.m_bytes < 0 or r.m_inp_bytes < 0:
            raise PlanError(ERR_TABLE, "cost table entries must be non-negative")
        prev = r.seq_len


def _row_for(table: CostTable, s: int) -> CostRow:
    """Profile group of a sequence: smallest tabulated length >= s."""
    for r in table.rows:
        if r.seq_len >= s:
            return r
    raise PlanError(ERR_TABLE, f"sequence length {s} exceeds the cost table")


@dataclass
class _Unit:
    tokens: int
    t_f: int
    t_b: int
    m: int
    m_inp: int


def _batch_units(seq_lens, batch_offsets, n_batches, table) -> List[_Unit]:
    units = []
    for i in range(n_batches):
        lo, hi = (i, i + 1) if batch_offsets is None else (batch_offsets[i], batch_offsets[i + 1])
        u = _Unit(0, 0, 0, 0, 0)
        for s in seq_lens[lo:hi]:
            r = _row_for(table, s)
            u.tokens = _fit(u.tokens + s)
            u.t_f = _fit(u.t_f + r.t_f_ns)
            u.t_b = _fit(u.t_b + r.t_b_ns)
            u.m = _fit(u.m + r.m_bytes)
            u.m_inp = _fit(u.m_inp + r.m_inp_bytes)
        units.append(u)
    return units


@dataclass
class _Cand:
    p: int
    b: int
    t_f: int
    t_b: int
    m: int
    m_inp: int
    M_bp: int


def _candidate(u: _Unit, p: int, b: int, L: int, M_C: int, o: PlanOpts) -> _Cand:
    """Costs of running b copies of the batch on p devices (one layer)."""
    if p == 1:
        c = 0
    else:
        vol = _fit(_fit(_fit(b * u.tokens) * o.hidden) * 2)
        per_link = _fit(_fit(p * p) * o.link_bytes_per_ns)
        c = _fit(4 * _fit(o.a2a_alpha_ns + _ceil_div(vol, per_link)))
    t_f = _fit(_ceil_div(_fit(b * u.t_f), p) + c)
    t_b = _fit(_ceil_div(_fit(b * u.t_b), p) + c)
    m = _ceil_div(_fit(b * u.m), p)
    m_inp = _ceil_div(_fit(b * u.m_inp), p)
    M_bp = _fit(_fit(L * m_inp) + M_C)  # Eq. (6) with r = L
    return _Cand(p, b, t_f, t_b, m, m_inp, M_bp)


def _step_time(c: _Cand, r: int, L: int, T_C: int) -> int:
    """Eqs. (4)-(5): L*t_f + L*t_b + r*t_f + T_C."""
    return _fit(_fit(_fit(L * _fit(c.t_f + c.t_b)) + _fit(r * c.t_f)) + T_C)


def _better(new, best, min_time: bool) -> bool:
    """Strictly better by Eq. (1) throughput b/(p*T) (or by raw time)."""
    if best is None:
        return True
    _, b1, p1, T1 = new
    _, b2, p2, T2 = best
    if min_time:
        return T1 < T2
    return b1 * p2 * T2 > b2 * p1 * T1


def _choose_config(u: _Unit, table: CostTable, budget: int, o: PlanOpts, batch_index: int):
    L, T_C, M_C = table.n_layers, table.T_C_ns, table.M_C_bytes
    best = None  # (cand, b, p, T) with r stored in cand tuple below
    best_r = None
    for p in o.sp_cands:
        if not (o.flags & FLAG_NO_HEAD_FILTER) and o.n_heads % p != 0:
            continue
        for b in range(1, o.b_max + 1):
            c = _candidate(u, p, b, L, M_C, o)
            if c.M_bp > budget:
                continue
            if o.mode == MODE_INTER:
                r = L
            else:
                # Algorithm 1: the smallest number of recomputed layers whose
                # stashed activations still fit, Eq. (6).
                # (exact integers: an unrepresentable total simply does not fit)
                r = None
                for rr in range(0, L + 1):
                    if (L - rr) * c.m + c.M_bp <= budget:
                        r = rr
                        break
                assert r is not None  # rr = L always fits once M_bp <= budget
            T = _step_time(c, r, L, T_C)
            key = (c, b, p, T)
            if _better(key, best, bool(o.flags & FLAG_MIN_TIME)):
                best, best_r = key, r
    if best is None:
        raise PlanError(ERR_INFEASIBLE, f"no feasible configuration for batch {batch_index}")
    c, b, p, T = best
    r = best_r
    mem = _fit(_fit((L - r) * c.m) + c.M_bp)
    return p, b, r, T, mem


def accumulation_steps(T: Sequence[int], g_min: int, g_max: int):
    """Eq. (3) with the bounds of Appendix C.

    Minimises sum_i (C - g_i*T_i) over accumulation vectors g whose iteration
    length C = max_j g_j*T_j stays within g_max * max_j T_j.  For a fixed C
    the best vector is g_i = floor(C / T_i) (each term is minimised on its
    own), and C itself is always some multiple k*T_j, so scanning those
    multiples visits every vector that can be optimal.  Ties go to the
    shortest iteration.  Returns ``(g, idle, makespan)`` after the G_min rule.
    """
    n = len(T)
    Tmax = max(T)
    bound = _fit(g_max * Tmax)
    count = 0
    for t in T:
        count += bound // t - _ceil_div(Tmax, t) + 1
    if count > MAX_ACCUM_CANDIDATES:
        raise PlanError(ERR_INVALID, "accumulation search too large")
    best = None
    for t in T:
        for kk in range(_ceil_div(Tmax, t), bound // t + 1):
            C = kk * t
            idle = sum(C - (C // ti) * ti for ti in T)
            if best is None or (idle, C) < best:
                best = (idle, C)
    C = best[1]
    g = [C // ti for ti in T]
    mg = max(g)
    if mg < g_min:
        f = _ceil_div(g_min, mg)
        g = [gi * f for gi in g]
    span = max(_fit(gi * ti) for gi, ti in zip(g, T))
    idle = _fit(sum(span - gi * ti for gi, ti in zip(g, T)))
    return g, idle, span


def plan(seq_lens: Sequence[int], table: CostTable, hbm_budget: int, opts: Optional[PlanOpts] = None,
         batch_offsets: Optional[Sequence[int]] = None, n_batches: Optional[int] = None) -> Plan:
    """Plan one training iteration.  Raises ``PlanError`` with a status code."""
    o = opts or PlanOpts()
    seq_lens = [int(s) for s in seq_lens]
    if n_batches is None:
        n_batches = len(seq_lens) if batch_offsets is None else len(batch_offsets) - 1
    if batch_offsets is not None:
        batch_offsets = [int(x) for x in batch_offsets]
    _validate(seq_lens, batch_offsets, n_batches, table, int(hbm_budget), o)
    units = _batch_units(seq_lens, batch_offsets, n_batches, table)
    out = Plan()
    L = table.n_layers
    for i, u in enumerate(units):
        p, b, r, T, mem = _choose_config(u, table, int(hbm_budget), o, i)
        out.sp_size.append(p)
        out.micro_batch.append(b)
        out.recompute_layers.append(r)
        out.step_time_ns.append(T)
        out.mem_bytes.append(mem)
        out.recompute_flags.extend(1 if layer < r else 0 for layer in range(L))
    if min(out.step_time_ns) == 0:
        raise PlanError(ERR_TABLE, "a batch has zero step time; the cost table is empty of cost")
    g, idle, span = accumulation_steps(out.step_time_ns, o.g_min, o.g_max)
    if max(g) > (1 << 31) - 1:
        raise PlanError(ERR_INVALID, "accumulation steps exceed int32")
    out.grad_accum = g
    out.idle_ns = idle
    out.makespan_ns = span
    return out


# --------------------------------------------------------------------------
# exhaustive searches used to pin the oracle (tests only)
# --------------------------------------------------------------------------

def brute_force_config(u_tokens, t_f1, t_b1, m1, m_inp1, table: CostTable, budget, o: PlanOpts):
    """Every (p, b, r) triple, checked directly against Eqs. (4)-(6).

    Returns the (p, b, r, T) maximising b/(p*T) (or minimising T with
    FLAG_MIN_TIME); ties: smaller p, smaller b, smaller r.  None if nothing
    fits.  Independent of ``_choose_config``: memory is evaluated for every r.
    """
    L, T_C, M_C = table.n_layers, table.T_C_ns, table.M_C_bytes
    best = None
    for p in sorted(o.sp_cands):
        if not (o.flags & FLAG_NO_HEAD_FILTER) and o.n_heads % p:
            continue
        for b in range(1, o.b_max + 1):
            comm = 0 if p == 1 else 4 * (o.a2a_alpha_ns + -(-(b * u_tokens * o.hidden * 2) // (p * p * o.link_bytes_per_ns)))
            tf = -(-(b * t_f1) // p) + comm
            tb = -(-(b * t_b1) // p) + comm
            m = -(-(b * m1) // p)
            mi = -(-(b * m_inp1) // p)
            rs = [L] if o.mode == MODE_INTER else range(L + 1)
            for r in rs:
                mem = (L - r) * m + L * mi + M_C
                if mem > budget:
                    continue
                T = L * tf + L * tb + r * tf + T_C
                if best is None:
                    best = (p, b, r, T)
                    continue
                bp, bb, br, bT = best
                if o.flags & FLAG_MIN_TIME:
                    better = T < bT
                else:
                    better = b * bp * bT > bb * p * T
                if better:
                    best = (p, b, r, T)
    return best


def brute_force_accumulation(T: Sequence[int], g_min: int, g_max: int):
    """Every g in prod_i [1, floor(g_max*max(T)/T_i)], scored by Eq. (3)."""
    bound = g_max * max(T)
    best = None
    for g in product(*[range(1, bound // t + 1) for t in T]):
        span = max(gi * ti for gi, ti in zip(g, T))
        idle = sum(span - gi * ti for gi, ti in zip(g, T))
        if best is None or (idle, span) < best[:2]:
            best = (idle, span, list(g))
    g = best[2]
    if max(g) < g_min:
        f = -(-g_min // max(g))
        g = [gi * f for gi in g]
    span = max(gi * ti for gi, ti in zip(g, T))
    idle = sum(span - gi * ti for gi, ti in zip(g, T))
    return g, idle, span
